// Generated: convolution variant e5m3_a4_o4. Do not edit.
#include "kernels.hpp"
#include "registry.hpp"
namespace hobflops {
namespace conv_e5m3_a4_o4 {
static __device__ __forceinline__ void mac_e5m3_a4(uint32_t (&acc)[12], const uint32_t (&w)[11], const uint32_t (&x)[11])
{
  const uint32_t acc_0 = acc[0];
  const uint32_t acc_1 = acc[1];
  const uint32_t acc_2 = acc[2];
  const uint32_t acc_3 = acc[3];
  const uint32_t acc_4 = acc[4];
  const uint32_t acc_5 = acc[5];
  const uint32_t acc_6 = acc[6];
  const uint32_t acc_7 = acc[7];
  const uint32_t acc_8 = acc[8];
  const uint32_t acc_9 = acc[9];
  const uint32_t acc_10 = acc[10];
  const uint32_t acc_11 = acc[11];
  const uint32_t w_0 = w[0];
  const uint32_t w_1 = w[1];
  const uint32_t w_2 = w[2];
  const uint32_t w_3 = w[3];
  const uint32_t w_4 = w[4];
  const uint32_t w_5 = w[5];
  const uint32_t w_6 = w[6];
  const uint32_t w_7 = w[7];
  const uint32_t w_8 = w[8];
  const uint32_t w_9 = w[9];
  const uint32_t w_10 = w[10];
  const uint32_t x_0 = x[0];
  const uint32_t x_1 = x[1];
  const uint32_t x_2 = x[2];
  const uint32_t x_3 = x[3];
  const uint32_t x_4 = x[4];
  const uint32_t x_5 = x[5];
  const uint32_t x_6 = x[6];
  const uint32_t x_7 = x[7];
  const uint32_t x_8 = x[8];
  const uint32_t x_9 = x[9];
  const uint32_t x_10 = x[10];
  const uint32_t t44 = (w_2 & x_0);
  const uint32_t t42 = (w_1 & x_1);
  const uint32_t t40 = (w_0 & x_2);
  const uint32_t t48 = __builtin_amdgcn_bitop3_b32(t44, t42, t40, 0xe8);
  const uint32_t t45 = (w_2 & x_1);
  const uint32_t t43 = (w_1 & x_2);
  const uint32_t t49 = __builtin_amdgcn_bitop3_b32(t45, t43, w_0, 0x96);
  const uint32_t t53 = __builtin_amdgcn_bitop3_b32(t49, t48, x_0, 0x96);
  const uint32_t t47 = __builtin_amdgcn_bitop3_b32(t44, t42, t40, 0x96);
  const uint32_t t41 = (w_1 & x_0);
  const uint32_t t60 = __builtin_amdgcn_bitop3_b32(t41, x_1, w_0, 0x80);
  const uint32_t t62 = (t47 & t60);
  const uint32_t t64 = (t53 & t62);
  const uint32_t t54 = __builtin_amdgcn_bitop3_b32(t49, t48, x_0, 0xe8);
  const uint32_t t50 = __builtin_amdgcn_bitop3_b32(t45, t43, w_0, 0xe8);
  const uint32_t t46 = (w_2 & x_2);
  const uint32_t t51 = __builtin_amdgcn_bitop3_b32(t46, x_1, w_1, 0x96);
  const uint32_t t57 = __builtin_amdgcn_bitop3_b32(t54, t51, t50, 0x96);
  const uint32_t t66 = (t57 & t64);
  const uint32_t t58 = __builtin_amdgcn_bitop3_b32(t54, t51, t50, 0xe8);
  const uint32_t t52 = __builtin_amdgcn_bitop3_b32(t46, x_1, w_1, 0xe8);
  const uint32_t t55 = __builtin_amdgcn_bitop3_b32(t52, x_2, w_2, 0x96);
  const uint32_t t68 = __builtin_amdgcn_bitop3_b32(t66, t58, t55, 0xe8);
  const uint32_t t56 = __builtin_amdgcn_bitop3_b32(t52, x_2, w_2, 0xe8);
  const uint32_t t69 = (t56 | t68);
  const uint32_t t59 = __builtin_amdgcn_bitop3_b32(t41, x_1, w_0, 0x78);
  const uint32_t t75 = (t59 & t69);
  const uint32_t t76 = __builtin_amdgcn_bitop3_b32(t75, x_0, w_0, 0xf8);
  const uint32_t t61 = (t47 ^ t60);
  const uint32_t t74 = __builtin_amdgcn_bitop3_b32(t69, t61, t59, 0xca);
  const uint32_t t63 = (t53 ^ t62);
  const uint32_t t70 = __builtin_amdgcn_bitop3_b32(t69, t63, t61, 0xca);
  const uint32_t t77 = __builtin_amdgcn_bitop3_b32(t76, t74, t70, 0x62);
  const uint32_t t116 = (~acc_0 & t77);
  const uint32_t t78 = (t70 & t74);
  const uint32_t t65 = (t57 ^ t64);
  const uint32_t t71 = __builtin_amdgcn_bitop3_b32(t69, t65, t63, 0xca);
  const uint32_t t79 = (t71 ^ t78);
  const uint32_t t117 = __builtin_amdgcn_bitop3_b32(t116, t79, acc_1, 0xd4);
  const uint32_t t80 = (t71 & t78);
  const uint32_t t67 = __builtin_amdgcn_bitop3_b32(t66, t58, t55, 0x96);
  const uint32_t t72 = __builtin_amdgcn_bitop3_b32(t69, t67, t65, 0xca);
  const uint32_t t81 = (t72 ^ t80);
  const uint32_t t118 = __builtin_amdgcn_bitop3_b32(t117, t81, acc_2, 0xd4);
  const uint32_t t82 = (t72 & t80);
  const uint32_t t73 = __builtin_amdgcn_bitop3_b32(t68, t67, t56, 0xa4);
  const uint32_t t83 = (t73 ^ t82);
  const uint32_t t119 = __builtin_amdgcn_bitop3_b32(t118, t83, acc_3, 0xd4);
  const uint32_t t84 = __builtin_amdgcn_bitop3_b32(t82, t73, t69, 0xea);
  const uint32_t t85 = __builtin_amdgcn_bitop3_b32(t84, x_3, w_3, 0x96);
  const uint32_t t120 = __builtin_amdgcn_bitop3_b32(t119, t85, acc_4, 0x8e);
  const uint32_t t86 = __builtin_amdgcn_bitop3_b32(t84, x_3, w_3, 0xe8);
  const uint32_t t87 = __builtin_amdgcn_bitop3_b32(t86, x_4, w_4, 0x96);
  const uint32_t t95 = (t85 ^ t87);
  const uint32_t t121 = __builtin_amdgcn_bitop3_b32(t120, t95, acc_5, 0xb2);
  const uint32_t t96 = (t85 & t87);
  const uint32_t t88 = __builtin_amdgcn_bitop3_b32(t86, x_4, w_4, 0xe8);
  const uint32_t t89 = __builtin_amdgcn_bitop3_b32(t88, x_5, w_5, 0x96);
  const uint32_t t97 = (t89 ^ t96);
  const uint32_t t122 = __builtin_amdgcn_bitop3_b32(t121, t97, acc_6, 0xb2);
  const uint32_t t98 = (t89 & t96);
  const uint32_t t90 = __builtin_amdgcn_bitop3_b32(t88, x_5, w_5, 0xe8);
  const uint32_t t91 = __builtin_amdgcn_bitop3_b32(t90, x_6, w_6, 0x96);
  const uint32_t t99 = (t91 ^ t98);
  const uint32_t t123 = __builtin_amdgcn_bitop3_b32(t122, t99, acc_7, 0xb2);
  const uint32_t t100 = (t91 & t98);
  const uint32_t t92 = __builtin_amdgcn_bitop3_b32(t90, x_6, w_6, 0xe8);
  const uint32_t t93 = __builtin_amdgcn_bitop3_b32(t92, x_7, w_7, 0x96);
  const uint32_t t101 = (t93 ^ t100);
  const uint32_t t124 = __builtin_amdgcn_bitop3_b32(t123, t101, acc_8, 0xe8);
  const uint32_t t102 = (t93 | t100);
  const uint32_t t94 = __builtin_amdgcn_bitop3_b32(t92, x_7, w_7, 0xe8);
  const uint32_t t103 = (t94 ^ t102);
  const uint32_t t36 = (~x_9 & x_10);
  const uint32_t t107 = __builtin_amdgcn_bitop3_b32(t36, w_10, w_9, 0x10);
  const uint32_t t37 = (x_9 | x_10);
  const uint32_t t106 = __builtin_amdgcn_bitop3_b32(t37, w_10, w_9, 0x04);
  const uint32_t t35 = (x_9 & x_10);
  const uint32_t t105 = __builtin_amdgcn_bitop3_b32(t35, w_10, w_9, 0xf8);
  const uint32_t t108 = __builtin_amdgcn_bitop3_b32(t107, t106, t105, 0xfe);
  const uint32_t t38 = (x_9 & ~x_10);
  const uint32_t t104 = __builtin_amdgcn_bitop3_b32(t38, w_10, w_9, 0x20);
  const uint32_t t112 = __builtin_amdgcn_bitop3_b32(t108, t104, t103, 0xf8);
  const uint32_t t125 = __builtin_amdgcn_bitop3_b32(t124, t112, acc_10, 0xb2);
  const uint32_t t147 = __builtin_amdgcn_bitop3_b32(t125, t85, acc_4, 0x18);
  const uint32_t t131 = __builtin_amdgcn_bitop3_b32(t125, t95, acc_5, 0xca);
  const uint32_t t127 = __builtin_amdgcn_bitop3_b32(t125, t95, acc_5, 0xac);
  const uint32_t t149 = __builtin_amdgcn_bitop3_b32(t147, t131, t127, 0xd4);
  const uint32_t t132 = __builtin_amdgcn_bitop3_b32(t125, t97, acc_6, 0xca);
  const uint32_t t128 = __builtin_amdgcn_bitop3_b32(t125, t97, acc_6, 0xac);
  const uint32_t t151 = __builtin_amdgcn_bitop3_b32(t149, t132, t128, 0xd4);
  const uint32_t t133 = __builtin_amdgcn_bitop3_b32(t125, t99, acc_7, 0xca);
  const uint32_t t129 = __builtin_amdgcn_bitop3_b32(t125, t99, acc_7, 0xac);
  const uint32_t t153 = __builtin_amdgcn_bitop3_b32(t151, t133, t129, 0xd4);
  const uint32_t t134 = __builtin_amdgcn_bitop3_b32(t125, t101, acc_8, 0x3a);
  const uint32_t t130 = __builtin_amdgcn_bitop3_b32(t125, t101, acc_8, 0x5c);
  const uint32_t t154 = __builtin_amdgcn_bitop3_b32(t153, t134, t130, 0x96);
  const uint32_t t152 = __builtin_amdgcn_bitop3_b32(t151, t133, t129, 0x96);
  const uint32_t t155 = (~t152 & t154);
  const uint32_t t144 = (acc_10 & t112);
  const uint32_t t156 = (t144 & t155);
  const uint32_t t142 = __builtin_amdgcn_bitop3_b32(t125, t83, acc_3, 0xca);
  const uint32_t t160 = (t142 & t156);
  const uint32_t t141 = __builtin_amdgcn_bitop3_b32(t125, t81, acc_2, 0xca);
  const uint32_t t159 = (t141 & t156);
  const uint32_t t146 = (acc_4 ^ t85);
  const uint32_t t164 = __builtin_amdgcn_bitop3_b32(t160, t159, t146, 0xd8);
  const uint32_t t140 = __builtin_amdgcn_bitop3_b32(t125, t79, acc_1, 0xca);
  const uint32_t t158 = (t140 & t156);
  const uint32_t t139 = __builtin_amdgcn_bitop3_b32(t125, t77, acc_0, 0xca);
  const uint32_t t157 = (t139 & t156);
  const uint32_t t162 = __builtin_amdgcn_bitop3_b32(t158, t157, t146, 0xd8);
  const uint32_t t148 = __builtin_amdgcn_bitop3_b32(t147, t131, t127, 0x96);
  const uint32_t t171 = __builtin_amdgcn_bitop3_b32(t164, t162, t148, 0xe4);
  const uint32_t t163 = __builtin_amdgcn_bitop3_b32(t159, t158, t146, 0xd8);
  const uint32_t t161 = (~t146 & t157);
  const uint32_t t170 = __builtin_amdgcn_bitop3_b32(t163, t161, t148, 0xe4);
  const uint32_t t169 = (t148 & t162);
  const uint32_t t176 = __builtin_amdgcn_bitop3_b32(t171, t170, t169, 0xfe);
  const uint32_t t165 = __builtin_amdgcn_bitop3_b32(t156, t146, t142, 0xb0);
  const uint32_t t172 = __builtin_amdgcn_bitop3_b32(t165, t163, t148, 0xe4);
  const uint32_t t150 = __builtin_amdgcn_bitop3_b32(t149, t132, t128, 0x96);
  const uint32_t t177 = __builtin_amdgcn_bitop3_b32(t176, t172, t150, 0xa8);
  const uint32_t t167 = (t148 & t161);
  const uint32_t t168 = __builtin_amdgcn_bitop3_b32(t167, t155, t144, 0xf2);
  const uint32_t t178 = (t168 | t177);
  const uint32_t t39 = (w_8 ^ x_8);
  const uint32_t t145 = (acc_9 ^ t39);
  const uint32_t t182 = (t145 & ~t178);
  const uint32_t t166 = (t146 & t156);
  const uint32_t t173 = __builtin_amdgcn_bitop3_b32(t166, t164, t148, 0xe4);
  const uint32_t t179 = __builtin_amdgcn_bitop3_b32(t173, t169, t150, 0xe4);
  const uint32_t t183 = (t145 ^ t179);
  const uint32_t t185 = (t182 & t183);
  const uint32_t t174 = (~t148 & t165);
  const uint32_t t180 = __builtin_amdgcn_bitop3_b32(t174, t170, t150, 0xe4);
  const uint32_t t186 = (t145 ^ t180);
  const uint32_t t188 = (t185 & t186);
  const uint32_t t175 = (~t148 & t166);
  const uint32_t t181 = __builtin_amdgcn_bitop3_b32(t175, t171, t150, 0xe4);
  const uint32_t t189 = (t145 ^ t181);
  const uint32_t t135 = __builtin_amdgcn_bitop3_b32(t125, t77, acc_0, 0xac);
  const uint32_t t191 = __builtin_amdgcn_bitop3_b32(t189, t188, t135, 0xe8);
  const uint32_t t192 = __builtin_amdgcn_bitop3_b32(t172, t150, t145, 0x9a);
  const uint32_t t136 = __builtin_amdgcn_bitop3_b32(t125, t79, acc_1, 0xac);
  const uint32_t t194 = __builtin_amdgcn_bitop3_b32(t192, t191, t136, 0xe8);
  const uint32_t t195 = __builtin_amdgcn_bitop3_b32(t173, t150, t145, 0x9a);
  const uint32_t t137 = __builtin_amdgcn_bitop3_b32(t125, t81, acc_2, 0xac);
  const uint32_t t197 = __builtin_amdgcn_bitop3_b32(t195, t194, t137, 0xe8);
  const uint32_t t198 = __builtin_amdgcn_bitop3_b32(t174, t150, t145, 0x9a);
  const uint32_t t138 = __builtin_amdgcn_bitop3_b32(t125, t83, acc_3, 0xac);
  const uint32_t t200 = __builtin_amdgcn_bitop3_b32(t198, t197, t138, 0xe8);
  const uint32_t t201 = __builtin_amdgcn_bitop3_b32(t175, t150, t145, 0x9a);
  const uint32_t t202 = (t200 ^ t201);
  const uint32_t t199 = __builtin_amdgcn_bitop3_b32(t198, t197, t138, 0x96);
  const uint32_t t196 = __builtin_amdgcn_bitop3_b32(t195, t194, t137, 0x96);
  const uint32_t t204 = __builtin_amdgcn_bitop3_b32(t202, t199, t196, 0x10);
  const uint32_t t203 = __builtin_amdgcn_bitop3_b32(t201, t200, t145, 0x54);
  const uint32_t t205 = (~t203 & t204);
  const uint32_t t190 = __builtin_amdgcn_bitop3_b32(t189, t188, t135, 0x96);
  const uint32_t t213 = __builtin_amdgcn_bitop3_b32(t205, t202, t190, 0x5c);
  const uint32_t t193 = __builtin_amdgcn_bitop3_b32(t192, t191, t136, 0x96);
  const uint32_t t214 = __builtin_amdgcn_bitop3_b32(t204, t203, t193, 0xec);
  const uint32_t t215 = (t213 & ~t214);
  const uint32_t t187 = (t185 ^ t186);
  const uint32_t t208 = (t187 & ~t205);
  const uint32_t t206 = (t178 & ~t205);
  const uint32_t t218 = __builtin_amdgcn_bitop3_b32(t215, t208, t206, 0xac);
  const uint32_t t184 = (t182 ^ t183);
  const uint32_t t207 = (t184 & ~t205);
  const uint32_t t217 = (t207 & ~t215);
  const uint32_t t212 = __builtin_amdgcn_bitop3_b32(t205, t199, t187, 0xac);
  const uint32_t t224 = __builtin_amdgcn_bitop3_b32(t214, t213, t212, 0xf8);
  const uint32_t t227 = __builtin_amdgcn_bitop3_b32(t224, t218, t217, 0xca);
  const uint32_t t216 = (t206 & ~t215);
  const uint32_t t226 = __builtin_amdgcn_bitop3_b32(t224, t217, t216, 0xca);
  const uint32_t t225 = (t216 & t224);
  const uint32_t t234 = __builtin_amdgcn_bitop3_b32(t227, t226, t225, 0xfe);
  const uint32_t t210 = __builtin_amdgcn_bitop3_b32(t205, t193, t178, 0xac);
  const uint32_t t220 = __builtin_amdgcn_bitop3_b32(t215, t210, t208, 0xac);
  const uint32_t t209 = (t190 & ~t205);
  const uint32_t t219 = __builtin_amdgcn_bitop3_b32(t215, t209, t207, 0xac);
  const uint32_t t229 = __builtin_amdgcn_bitop3_b32(t224, t220, t219, 0xca);
  const uint32_t t228 = __builtin_amdgcn_bitop3_b32(t224, t219, t218, 0xca);
  const uint32_t t235 = __builtin_amdgcn_bitop3_b32(t234, t229, t228, 0x64);
  const uint32_t t236 = (t228 & t229);
  const uint32_t t211 = __builtin_amdgcn_bitop3_b32(t205, t196, t184, 0xac);
  const uint32_t t221 = __builtin_amdgcn_bitop3_b32(t215, t211, t209, 0xac);
  const uint32_t t230 = __builtin_amdgcn_bitop3_b32(t224, t221, t220, 0xca);
  const uint32_t t237 = (t230 ^ t236);
  const uint32_t t238 = (t230 & t236);
  const uint32_t t222 = __builtin_amdgcn_bitop3_b32(t215, t212, t210, 0xac);
  const uint32_t t231 = __builtin_amdgcn_bitop3_b32(t224, t222, t221, 0xca);
  const uint32_t t239 = (t231 ^ t238);
  const uint32_t t240 = (t231 & t238);
  const uint32_t t223 = __builtin_amdgcn_bitop3_b32(t214, t213, t211, 0xc4);
  const uint32_t t232 = __builtin_amdgcn_bitop3_b32(t224, t223, t222, 0x3a);
  const uint32_t t241 = (t232 ^ t240);
  const uint32_t t242 = (t232 & t240);
  const uint32_t t126 = __builtin_amdgcn_bitop3_b32(t125, t85, acc_4, 0x5c);
  const uint32_t t245 = __builtin_amdgcn_bitop3_b32(t242, t224, t126, 0x69);
  const uint32_t t246 = __builtin_amdgcn_bitop3_b32(t242, t224, t126, 0xd4);
  const uint32_t t247 = __builtin_amdgcn_bitop3_b32(t246, t215, t127, 0x96);
  const uint32_t t248 = __builtin_amdgcn_bitop3_b32(t246, t215, t127, 0xe8);
  const uint32_t t243 = (t205 ^ t215);
  const uint32_t t249 = __builtin_amdgcn_bitop3_b32(t248, t243, t128, 0x96);
  const uint32_t t250 = __builtin_amdgcn_bitop3_b32(t248, t243, t128, 0xe8);
  const uint32_t t244 = (t205 | t215);
  const uint32_t t251 = __builtin_amdgcn_bitop3_b32(t250, t244, t129, 0x96);
  const uint32_t t252 = __builtin_amdgcn_bitop3_b32(t250, t244, t129, 0xe8);
  const uint32_t t253 = __builtin_amdgcn_bitop3_b32(t252, t244, t130, 0x69);
  const uint32_t t233 = (t223 & ~t224);
  const uint32_t t143 = __builtin_amdgcn_bitop3_b32(t125, t39, acc_9, 0xac);
  const uint32_t t265 = (t143 & ~t233);
  const uint32_t t256 = (acc_10 | t112);
  const uint32_t t264 = (acc_9 & t39);
  const uint32_t t266 = __builtin_amdgcn_bitop3_b32(t265, t264, t256, 0xe4);
  const uint32_t t110 = __builtin_amdgcn_bitop3_b32(t104, t102, t94, 0x80);
  const uint32_t t109 = __builtin_amdgcn_bitop3_b32(t36, w_10, w_9, 0xf4);
  const uint32_t t111 = __builtin_amdgcn_bitop3_b32(t110, t109, t108, 0xfe);
  const uint32_t t115 = (t111 & ~t112);
  const uint32_t t113 = (~acc_10 & acc_11);
  const uint32_t t261 = (t113 | t115);
  const uint32_t t267 = __builtin_amdgcn_bitop3_b32(t113, t39, acc_9, 0xac);
  const uint32_t t268 = __builtin_amdgcn_bitop3_b32(t267, t266, t261, 0xe4);
  const uint32_t t254 = __builtin_amdgcn_bitop3_b32(t252, t244, t130, 0xd4);
  const uint32_t t255 = (t244 ^ t254);
  const uint32_t t257 = __builtin_amdgcn_bitop3_b32(t256, t111, acc_11, 0x10);
  const uint32_t t262 = (~t233 & t257);
  const uint32_t t259 = __builtin_amdgcn_bitop3_b32(t145, t115, t113, 0x80);
  const uint32_t t114 = (t111 & t112);
  const uint32_t t258 = __builtin_amdgcn_bitop3_b32(t114, acc_11, acc_10, 0xf8);
  const uint32_t t260 = (t258 | t259);
  const uint32_t t270 = __builtin_amdgcn_bitop3_b32(t262, t260, t255, 0xdc);
  const uint32_t t263 = __builtin_amdgcn_bitop3_b32(t262, t254, t244, 0x40);
  const uint32_t t269 = __builtin_amdgcn_bitop3_b32(t263, t261, t260, 0xfe);
  acc[0] = t235;
  acc[1] = t237;
  acc[2] = t239;
  acc[3] = t241;
  acc[4] = t245;
  acc[5] = t247;
  acc[6] = t249;
  acc[7] = t251;
  acc[8] = t253;
  acc[9] = t268;
  acc[10] = t270;
  acc[11] = t269;
}

static __device__ __forceinline__ void epi_e5m4_o4(const uint32_t (&a)[12], uint32_t (&r)[12])
{
  const uint32_t a_0 = a[0];
  const uint32_t a_1 = a[1];
  const uint32_t a_2 = a[2];
  const uint32_t a_3 = a[3];
  const uint32_t a_4 = a[4];
  const uint32_t a_5 = a[5];
  const uint32_t a_6 = a[6];
  const uint32_t a_7 = a[7];
  const uint32_t a_8 = a[8];
  const uint32_t a_9 = a[9];
  const uint32_t a_10 = a[10];
  const uint32_t a_11 = a[11];
  const uint32_t t13 = __builtin_amdgcn_bitop3_b32(a_11, a_10, a_0, 0x08);
  const uint32_t t14 = __builtin_amdgcn_bitop3_b32(a_11, a_10, a_1, 0x08);
  const uint32_t t15 = __builtin_amdgcn_bitop3_b32(a_11, a_10, a_2, 0x08);
  const uint32_t t16 = __builtin_amdgcn_bitop3_b32(a_11, a_10, a_3, 0x08);
  const uint32_t t17 = __builtin_amdgcn_bitop3_b32(a_11, a_10, a_4, 0x08);
  const uint32_t t18 = __builtin_amdgcn_bitop3_b32(a_11, a_10, a_5, 0x08);
  const uint32_t t19 = __builtin_amdgcn_bitop3_b32(a_11, a_10, a_6, 0x08);
  const uint32_t t20 = __builtin_amdgcn_bitop3_b32(a_11, a_10, a_7, 0x08);
  const uint32_t t21 = __builtin_amdgcn_bitop3_b32(a_11, a_10, a_8, 0x08);
  const uint32_t t22 = __builtin_amdgcn_bitop3_b32(a_11, a_10, a_9, 0x2a);
  r[0] = t13;
  r[1] = t14;
  r[2] = t15;
  r[3] = t16;
  r[4] = t17;
  r[5] = t18;
  r[6] = t19;
  r[7] = t20;
  r[8] = t21;
  r[9] = t22;
  r[10] = a_10;
  r[11] = a_11;
}

static __device__ __forceinline__ void prod_e5m3_a4(const uint32_t (&w)[11], const uint32_t (&x)[11], uint32_t (&p)[12])
{
  const uint32_t w_0 = w[0];
  const uint32_t w_1 = w[1];
  const uint32_t w_2 = w[2];
  const uint32_t w_3 = w[3];
  const uint32_t w_4 = w[4];
  const uint32_t w_5 = w[5];
  const uint32_t w_6 = w[6];
  const uint32_t w_7 = w[7];
  const uint32_t w_8 = w[8];
  const uint32_t w_9 = w[9];
  const uint32_t w_10 = w[10];
  const uint32_t x_0 = x[0];
  const uint32_t x_1 = x[1];
  const uint32_t x_2 = x[2];
  const uint32_t x_3 = x[3];
  const uint32_t x_4 = x[4];
  const uint32_t x_5 = x[5];
  const uint32_t x_6 = x[6];
  const uint32_t x_7 = x[7];
  const uint32_t x_8 = x[8];
  const uint32_t x_9 = x[9];
  const uint32_t x_10 = x[10];
  const uint32_t t32 = (w_2 & x_0);
  const uint32_t t30 = (w_1 & x_1);
  const uint32_t t28 = (w_0 & x_2);
  const uint32_t t36 = __builtin_amdgcn_bitop3_b32(t32, t30, t28, 0xe8);
  const uint32_t t33 = (w_2 & x_1);
  const uint32_t t31 = (w_1 & x_2);
  const uint32_t t37 = __builtin_amdgcn_bitop3_b32(t33, t31, w_0, 0x96);
  const uint32_t t41 = __builtin_amdgcn_bitop3_b32(t37, t36, x_0, 0x96);
  const uint32_t t35 = __builtin_amdgcn_bitop3_b32(t32, t30, t28, 0x96);
  const uint32_t t29 = (w_1 & x_0);
  const uint32_t t48 = __builtin_amdgcn_bitop3_b32(t29, x_1, w_0, 0x80);
  const uint32_t t50 = (t35 & t48);
  const uint32_t t52 = (t41 & t50);
  const uint32_t t42 = __builtin_amdgcn_bitop3_b32(t37, t36, x_0, 0xe8);
  const uint32_t t38 = __builtin_amdgcn_bitop3_b32(t33, t31, w_0, 0xe8);
  const uint32_t t34 = (w_2 & x_2);
  const uint32_t t39 = __builtin_amdgcn_bitop3_b32(t34, x_1, w_1, 0x96);
  const uint32_t t45 = __builtin_amdgcn_bitop3_b32(t42, t39, t38, 0x96);
  const uint32_t t54 = (t45 & t52);
  const uint32_t t46 = __builtin_amdgcn_bitop3_b32(t42, t39, t38, 0xe8);
  const uint32_t t40 = __builtin_amdgcn_bitop3_b32(t34, x_1, w_1, 0xe8);
  const uint32_t t43 = __builtin_amdgcn_bitop3_b32(t40, x_2, w_2, 0x96);
  const uint32_t t56 = __builtin_amdgcn_bitop3_b32(t54, t46, t43, 0xe8);
  const uint32_t t44 = __builtin_amdgcn_bitop3_b32(t40, x_2, w_2, 0xe8);
  const uint32_t t57 = (t44 | t56);
  const uint32_t t47 = __builtin_amdgcn_bitop3_b32(t29, x_1, w_0, 0x78);
  const uint32_t t63 = (t47 & t57);
  const uint32_t t64 = __builtin_amdgcn_bitop3_b32(t63, x_0, w_0, 0xf8);
  const uint32_t t49 = (t35 ^ t48);
  const uint32_t t62 = __builtin_amdgcn_bitop3_b32(t57, t49, t47, 0xca);
  const uint32_t t51 = (t41 ^ t50);
  const uint32_t t58 = __builtin_amdgcn_bitop3_b32(t57, t51, t49, 0xca);
  const uint32_t t65 = __builtin_amdgcn_bitop3_b32(t64, t62, t58, 0x62);
  const uint32_t t66 = (t58 & t62);
  const uint32_t t53 = (t45 ^ t52);
  const uint32_t t59 = __builtin_amdgcn_bitop3_b32(t57, t53, t51, 0xca);
  const uint32_t t67 = (t59 ^ t66);
  const uint32_t t68 = (t59 & t66);
  const uint32_t t55 = __builtin_amdgcn_bitop3_b32(t54, t46, t43, 0x96);
  const uint32_t t60 = __builtin_amdgcn_bitop3_b32(t57, t55, t53, 0xca);
  const uint32_t t69 = (t60 ^ t68);
  const uint32_t t70 = (t60 & t68);
  const uint32_t t61 = __builtin_amdgcn_bitop3_b32(t56, t55, t44, 0xa4);
  const uint32_t t71 = (t61 ^ t70);
  const uint32_t t72 = __builtin_amdgcn_bitop3_b32(t70, t61, t57, 0xea);
  const uint32_t t73 = __builtin_amdgcn_bitop3_b32(t72, x_3, w_3, 0x69);
  const uint32_t t74 = __builtin_amdgcn_bitop3_b32(t72, x_3, w_3, 0xe8);
  const uint32_t t75 = __builtin_amdgcn_bitop3_b32(t74, x_4, w_4, 0x96);
  const uint32_t t83 = ~(t73 ^ t75);
  const uint32_t t84 = (~t73 & t75);
  const uint32_t t76 = __builtin_amdgcn_bitop3_b32(t74, x_4, w_4, 0xe8);
  const uint32_t t77 = __builtin_amdgcn_bitop3_b32(t76, x_5, w_5, 0x96);
  const uint32_t t85 = (t77 ^ t84);
  const uint32_t t86 = (t77 & t84);
  const uint32_t t78 = __builtin_amdgcn_bitop3_b32(t76, x_5, w_5, 0xe8);
  const uint32_t t79 = __builtin_amdgcn_bitop3_b32(t78, x_6, w_6, 0x96);
  const uint32_t t87 = (t79 ^ t86);
  const uint32_t t88 = (t79 & t86);
  const uint32_t t80 = __builtin_amdgcn_bitop3_b32(t78, x_6, w_6, 0xe8);
  const uint32_t t81 = __builtin_amdgcn_bitop3_b32(t80, x_7, w_7, 0x96);
  const uint32_t t89 = ~(t81 ^ t88);
  const uint32_t t27 = (w_8 ^ x_8);
  const uint32_t t90 = (t81 | t88);
  const uint32_t t82 = __builtin_amdgcn_bitop3_b32(t80, x_7, w_7, 0xe8);
  const uint32_t t91 = (t82 ^ t90);
  const uint32_t t24 = (~x_9 & x_10);
  const uint32_t t95 = __builtin_amdgcn_bitop3_b32(t24, w_10, w_9, 0x10);
  const uint32_t t25 = (x_9 | x_10);
  const uint32_t t94 = __builtin_amdgcn_bitop3_b32(t25, w_10, w_9, 0x04);
  const uint32_t t23 = (x_9 & x_10);
  const uint32_t t93 = __builtin_amdgcn_bitop3_b32(t23, w_10, w_9, 0xf8);
  const uint32_t t96 = __builtin_amdgcn_bitop3_b32(t95, t94, t93, 0xfe);
  const uint32_t t26 = (x_9 & ~x_10);
  const uint32_t t92 = __builtin_amdgcn_bitop3_b32(t26, w_10, w_9, 0x20);
  const uint32_t t100 = __builtin_amdgcn_bitop3_b32(t96, t92, t91, 0xf8);
  const uint32_t t98 = __builtin_amdgcn_bitop3_b32(t92, t90, t82, 0x80);
  const uint32_t t97 = __builtin_amdgcn_bitop3_b32(t24, w_10, w_9, 0xf4);
  const uint32_t t99 = __builtin_amdgcn_bitop3_b32(t98, t97, t96, 0xfe);
  p[0] = t65;
  p[1] = t67;
  p[2] = t69;
  p[3] = t71;
  p[4] = t73;
  p[5] = t83;
  p[6] = t85;
  p[7] = t87;
  p[8] = t89;
  p[9] = t27;
  p[10] = t100;
  p[11] = t99;
}

static __device__ __forceinline__ void accum_e5m4(uint32_t (&acc)[12], const uint32_t (&p)[12])
{
  const uint32_t acc_0 = acc[0];
  const uint32_t acc_1 = acc[1];
  const uint32_t acc_2 = acc[2];
  const uint32_t acc_3 = acc[3];
  const uint32_t acc_4 = acc[4];
  const uint32_t acc_5 = acc[5];
  const uint32_t acc_6 = acc[6];
  const uint32_t acc_7 = acc[7];
  const uint32_t acc_8 = acc[8];
  const uint32_t acc_9 = acc[9];
  const uint32_t acc_10 = acc[10];
  const uint32_t acc_11 = acc[11];
  const uint32_t p_0 = p[0];
  const uint32_t p_1 = p[1];
  const uint32_t p_2 = p[2];
  const uint32_t p_3 = p[3];
  const uint32_t p_4 = p[4];
  const uint32_t p_5 = p[5];
  const uint32_t p_6 = p[6];
  const uint32_t p_7 = p[7];
  const uint32_t p_8 = p[8];
  const uint32_t p_9 = p[9];
  const uint32_t p_10 = p[10];
  const uint32_t p_11 = p[11];
  const uint32_t t27 = (~acc_0 & p_0);
  const uint32_t t28 = __builtin_amdgcn_bitop3_b32(t27, p_1, acc_1, 0xd4);
  const uint32_t t29 = __builtin_amdgcn_bitop3_b32(t28, p_2, acc_2, 0xd4);
  const uint32_t t30 = __builtin_amdgcn_bitop3_b32(t29, p_3, acc_3, 0xd4);
  const uint32_t t31 = __builtin_amdgcn_bitop3_b32(t30, p_4, acc_4, 0xd4);
  const uint32_t t32 = __builtin_amdgcn_bitop3_b32(t31, p_5, acc_5, 0xd4);
  const uint32_t t33 = __builtin_amdgcn_bitop3_b32(t32, p_6, acc_6, 0xd4);
  const uint32_t t34 = __builtin_amdgcn_bitop3_b32(t33, p_7, acc_7, 0xd4);
  const uint32_t t35 = __builtin_amdgcn_bitop3_b32(t34, p_8, acc_8, 0xd4);
  const uint32_t t36 = __builtin_amdgcn_bitop3_b32(t35, p_10, acc_10, 0xd4);
  const uint32_t t57 = __builtin_amdgcn_bitop3_b32(t36, p_4, acc_4, 0x24);
  const uint32_t t42 = __builtin_amdgcn_bitop3_b32(t36, p_5, acc_5, 0xac);
  const uint32_t t38 = __builtin_amdgcn_bitop3_b32(t36, p_5, acc_5, 0xca);
  const uint32_t t59 = __builtin_amdgcn_bitop3_b32(t57, t42, t38, 0xd4);
  const uint32_t t43 = __builtin_amdgcn_bitop3_b32(t36, p_6, acc_6, 0xac);
  const uint32_t t39 = __builtin_amdgcn_bitop3_b32(t36, p_6, acc_6, 0xca);
  const uint32_t t61 = __builtin_amdgcn_bitop3_b32(t59, t43, t39, 0xd4);
  const uint32_t t44 = __builtin_amdgcn_bitop3_b32(t36, p_7, acc_7, 0xac);
  const uint32_t t40 = __builtin_amdgcn_bitop3_b32(t36, p_7, acc_7, 0xca);
  const uint32_t t63 = __builtin_amdgcn_bitop3_b32(t61, t44, t40, 0xd4);
  const uint32_t t45 = __builtin_amdgcn_bitop3_b32(t36, p_8, acc_8, 0xac);
  const uint32_t t41 = __builtin_amdgcn_bitop3_b32(t36, p_8, acc_8, 0xca);
  const uint32_t t64 = __builtin_amdgcn_bitop3_b32(t63, t45, t41, 0x96);
  const uint32_t t62 = __builtin_amdgcn_bitop3_b32(t61, t44, t40, 0x96);
  const uint32_t t65 = (t62 | t64);
  const uint32_t t66 = __builtin_amdgcn_bitop3_b32(t65, p_10, acc_10, 0x08);
  const uint32_t t53 = __builtin_amdgcn_bitop3_b32(t36, p_3, acc_3, 0xac);
  const uint32_t t70 = (t53 & t66);
  const uint32_t t52 = __builtin_amdgcn_bitop3_b32(t36, p_2, acc_2, 0xac);
  const uint32_t t69 = (t52 & t66);
  const uint32_t t56 = (acc_4 ^ p_4);
  const uint32_t t75 = __builtin_amdgcn_bitop3_b32(t70, t69, t56, 0xe4);
  const uint32_t t51 = __builtin_amdgcn_bitop3_b32(t36, p_1, acc_1, 0xac);
  const uint32_t t68 = (t51 & t66);
  const uint32_t t50 = __builtin_amdgcn_bitop3_b32(t36, p_0, acc_0, 0xac);
  const uint32_t t67 = (t50 & t66);
  const uint32_t t73 = __builtin_amdgcn_bitop3_b32(t68, t67, t56, 0xe4);
  const uint32_t t58 = __builtin_amdgcn_bitop3_b32(t57, t42, t38, 0x96);
  const uint32_t t81 = __builtin_amdgcn_bitop3_b32(t75, t73, t58, 0xe4);
  const uint32_t t74 = __builtin_amdgcn_bitop3_b32(t69, t68, t56, 0xe4);
  const uint32_t t72 = (t56 & t67);
  const uint32_t t80 = __builtin_amdgcn_bitop3_b32(t74, t72, t58, 0xe4);
  const uint32_t t79 = (t58 & t73);
  const uint32_t t86 = __builtin_amdgcn_bitop3_b32(t81, t80, t79, 0xfe);
  const uint32_t t76 = __builtin_amdgcn_bitop3_b32(t66, t56, t53, 0xe0);
  const uint32_t t82 = __builtin_amdgcn_bitop3_b32(t76, t74, t58, 0xe4);
  const uint32_t t60 = __builtin_amdgcn_bitop3_b32(t59, t43, t39, 0x96);
  const uint32_t t87 = __builtin_amdgcn_bitop3_b32(t86, t82, t60, 0xa8);
  const uint32_t t71 = __builtin_amdgcn_bitop3_b32(t65, p_10, acc_10, 0x80);
  const uint32_t t78 = __builtin_amdgcn_bitop3_b32(t72, t71, t58, 0xec);
  const uint32_t t88 = (t78 | t87);
  const uint32_t t55 = (acc_9 ^ p_9);
  const uint32_t t92 = (t55 & ~t88);
  const uint32_t t77 = (~t56 & t66);
  const uint32_t t83 = __builtin_amdgcn_bitop3_b32(t77, t75, t58, 0xe4);
  const uint32_t t89 = __builtin_amdgcn_bitop3_b32(t83, t79, t60, 0xe4);
  const uint32_t t93 = (t55 ^ t89);
  const uint32_t t95 = (t92 & t93);
  const uint32_t t84 = (~t58 & t76);
  const uint32_t t90 = __builtin_amdgcn_bitop3_b32(t84, t80, t60, 0xe4);
  const uint32_t t96 = (t55 ^ t90);
  const uint32_t t98 = (t95 & t96);
  const uint32_t t85 = (~t58 & t77);
  const uint32_t t91 = __builtin_amdgcn_bitop3_b32(t85, t81, t60, 0xe4);
  const uint32_t t99 = (t55 ^ t91);
  const uint32_t t46 = __builtin_amdgcn_bitop3_b32(t36, p_0, acc_0, 0xca);
  const uint32_t t101 = __builtin_amdgcn_bitop3_b32(t99, t98, t46, 0xe8);
  const uint32_t t102 = __builtin_amdgcn_bitop3_b32(t82, t60, t55, 0x9a);
  const uint32_t t47 = __builtin_amdgcn_bitop3_b32(t36, p_1, acc_1, 0xca);
  const uint32_t t104 = __builtin_amdgcn_bitop3_b32(t102, t101, t47, 0xe8);
  const uint32_t t105 = __builtin_amdgcn_bitop3_b32(t83, t60, t55, 0x9a);
  const uint32_t t48 = __builtin_amdgcn_bitop3_b32(t36, p_2, acc_2, 0xca);
  const uint32_t t107 = __builtin_amdgcn_bitop3_b32(t105, t104, t48, 0xe8);
  const uint32_t t108 = __builtin_amdgcn_bitop3_b32(t84, t60, t55, 0x9a);
  const uint32_t t49 = __builtin_amdgcn_bitop3_b32(t36, p_3, acc_3, 0xca);
  const uint32_t t110 = __builtin_amdgcn_bitop3_b32(t108, t107, t49, 0xe8);
  const uint32_t t111 = __builtin_amdgcn_bitop3_b32(t85, t60, t55, 0x9a);
  const uint32_t t112 = (t110 ^ t111);
  const uint32_t t109 = __builtin_amdgcn_bitop3_b32(t108, t107, t49, 0x96);
  const uint32_t t106 = __builtin_amdgcn_bitop3_b32(t105, t104, t48, 0x96);
  const uint32_t t114 = __builtin_amdgcn_bitop3_b32(t112, t109, t106, 0x10);
  const uint32_t t113 = __builtin_amdgcn_bitop3_b32(t111, t110, t55, 0x54);
  const uint32_t t115 = (~t113 & t114);
  const uint32_t t100 = __builtin_amdgcn_bitop3_b32(t99, t98, t46, 0x96);
  const uint32_t t123 = __builtin_amdgcn_bitop3_b32(t115, t112, t100, 0x5c);
  const uint32_t t103 = __builtin_amdgcn_bitop3_b32(t102, t101, t47, 0x96);
  const uint32_t t124 = __builtin_amdgcn_bitop3_b32(t114, t113, t103, 0xec);
  const uint32_t t125 = (t123 & ~t124);
  const uint32_t t97 = (t95 ^ t96);
  const uint32_t t118 = (t97 & ~t115);
  const uint32_t t116 = (t88 & ~t115);
  const uint32_t t128 = __builtin_amdgcn_bitop3_b32(t125, t118, t116, 0xac);
  const uint32_t t94 = (t92 ^ t93);
  const uint32_t t117 = (t94 & ~t115);
  const uint32_t t127 = (t117 & ~t125);
  const uint32_t t122 = __builtin_amdgcn_bitop3_b32(t115, t109, t97, 0xac);
  const uint32_t t134 = __builtin_amdgcn_bitop3_b32(t124, t123, t122, 0xf8);
  const uint32_t t137 = __builtin_amdgcn_bitop3_b32(t134, t128, t127, 0xca);
  const uint32_t t126 = (t116 & ~t125);
  const uint32_t t136 = __builtin_amdgcn_bitop3_b32(t134, t127, t126, 0xca);
  const uint32_t t135 = (t126 & t134);
  const uint32_t t144 = __builtin_amdgcn_bitop3_b32(t137, t136, t135, 0xfe);
  const uint32_t t120 = __builtin_amdgcn_bitop3_b32(t115, t103, t88, 0xac);
  const uint32_t t130 = __builtin_amdgcn_bitop3_b32(t125, t120, t118, 0xac);
  const uint32_t t119 = (t100 & ~t115);
  const uint32_t t129 = __builtin_amdgcn_bitop3_b32(t125, t119, t117, 0xac);
  const uint32_t t139 = __builtin_amdgcn_bitop3_b32(t134, t130, t129, 0xca);
  const uint32_t t138 = __builtin_amdgcn_bitop3_b32(t134, t129, t128, 0xca);
  const uint32_t t145 = __builtin_amdgcn_bitop3_b32(t144, t139, t138, 0x64);
  const uint32_t t146 = (t138 & t139);
  const uint32_t t121 = __builtin_amdgcn_bitop3_b32(t115, t106, t94, 0xac);
  const uint32_t t131 = __builtin_amdgcn_bitop3_b32(t125, t121, t119, 0xac);
  const uint32_t t140 = __builtin_amdgcn_bitop3_b32(t134, t131, t130, 0xca);
  const uint32_t t147 = (t140 ^ t146);
  const uint32_t t148 = (t140 & t146);
  const uint32_t t132 = __builtin_amdgcn_bitop3_b32(t125, t122, t120, 0xac);
  const uint32_t t141 = __builtin_amdgcn_bitop3_b32(t134, t132, t131, 0xca);
  const uint32_t t149 = (t141 ^ t148);
  const uint32_t t150 = (t141 & t148);
  const uint32_t t133 = __builtin_amdgcn_bitop3_b32(t124, t123, t121, 0xc4);
  const uint32_t t142 = __builtin_amdgcn_bitop3_b32(t134, t133, t132, 0x3a);
  const uint32_t t151 = (t142 ^ t150);
  const uint32_t t152 = (t142 & t150);
  const uint32_t t37 = __builtin_amdgcn_bitop3_b32(t36, p_4, acc_4, 0xca);
  const uint32_t t155 = __builtin_amdgcn_bitop3_b32(t152, t134, t37, 0x96);
  const uint32_t t156 = __builtin_amdgcn_bitop3_b32(t152, t134, t37, 0xe8);
  const uint32_t t157 = __builtin_amdgcn_bitop3_b32(t156, t125, t38, 0x96);
  const uint32_t t158 = __builtin_amdgcn_bitop3_b32(t156, t125, t38, 0xe8);
  const uint32_t t153 = (t115 ^ t125);
  const uint32_t t159 = __builtin_amdgcn_bitop3_b32(t158, t153, t39, 0x96);
  const uint32_t t160 = __builtin_amdgcn_bitop3_b32(t158, t153, t39, 0xe8);
  const uint32_t t154 = (t115 | t125);
  const uint32_t t161 = __builtin_amdgcn_bitop3_b32(t160, t154, t40, 0x96);
  const uint32_t t162 = __builtin_amdgcn_bitop3_b32(t160, t154, t40, 0xe8);
  const uint32_t t163 = __builtin_amdgcn_bitop3_b32(t162, t154, t41, 0x96);
  const uint32_t t143 = (t133 & ~t134);
  const uint32_t t54 = __builtin_amdgcn_bitop3_b32(t36, p_9, acc_9, 0xca);
  const uint32_t t175 = (t54 & ~t143);
  const uint32_t t174 = (acc_9 & p_9);
  const uint32_t t166 = (acc_10 | p_10);
  const uint32_t t176 = __builtin_amdgcn_bitop3_b32(t175, t174, t166, 0xe4);
  const uint32_t t25 = (~acc_10 & acc_11);
  const uint32_t t177 = __builtin_amdgcn_bitop3_b32(t25, p_9, acc_9, 0xac);
  const uint32_t t171 = __builtin_amdgcn_bitop3_b32(t25, p_11, p_10, 0xf4);
  const uint32_t t178 = __builtin_amdgcn_bitop3_b32(t177, t176, t171, 0xe4);
  const uint32_t t164 = __builtin_amdgcn_bitop3_b32(t162, t154, t41, 0xe8);
  const uint32_t t165 = (t154 ^ t164);
  const uint32_t t167 = __builtin_amdgcn_bitop3_b32(t166, p_11, acc_11, 0x10);
  const uint32_t t172 = (~t143 & t167);
  const uint32_t t169 = __builtin_amdgcn_bitop3_b32(t25, p_11, p_10, 0x40);
  const uint32_t t26 = (p_10 & p_11);
  const uint32_t t168 = __builtin_amdgcn_bitop3_b32(t26, acc_11, acc_10, 0xf8);
  const uint32_t t170 = __builtin_amdgcn_bitop3_b32(t169, t168, t55, 0xec);
  const uint32_t t180 = __builtin_amdgcn_bitop3_b32(t172, t170, t165, 0xdc);
  const uint32_t t173 = __builtin_amdgcn_bitop3_b32(t172, t164, t154, 0x40);
  const uint32_t t179 = __builtin_amdgcn_bitop3_b32(t173, t171, t170, 0xfe);
  acc[0] = t145;
  acc[1] = t147;
  acc[2] = t149;
  acc[3] = t151;
  acc[4] = t155;
  acc[5] = t157;
  acc[6] = t159;
  acc[7] = t161;
  acc[8] = t163;
  acc[9] = t178;
  acc[10] = t180;
  acc[11] = t179;
}

static constexpr int kAccSlot[12] = {0, 1, 5, 3, 2, 9, 6, 7, 10, 11, 4, 8};
static constexpr int kProdSlot[12] = {0, 2, 6, 1, 3, 10, 5, 9, 7, 4, 11, 8};
// Adds the K products of one batch into acc (planes in register-slot order).
static __device__ __forceinline__ void accum_batch(uint32_t (&acc)[12], const lds_u32* entry) {
  asm volatile(
      "s_waitcnt lgkmcnt(0)\n"
      "ds_read_b128 v[120:123], %[e] offset:0\n"
      "ds_read_b128 v[124:127], %[e] offset:16\n"
      "ds_read_b128 v[128:131], %[e] offset:32\n"
      "ds_read_b128 v[132:135], %[e] offset:12288\n"
      "ds_read_b128 v[136:139], %[e] offset:12304\n"
      "ds_read_b128 v[140:143], %[e] offset:12320\n"
      "ds_read_b128 v[144:147], %[e] offset:24576\n"
      "ds_read_b128 v[148:151], %[e] offset:24592\n"
      "ds_read_b128 v[152:155], %[e] offset:24608\n"
      "ds_read_b128 v[156:159], %[e] offset:36864\n"
      "ds_read_b128 v[160:163], %[e] offset:36880\n"
      "ds_read_b128 v[164:167], %[e] offset:36896\n"
      "s_waitcnt lgkmcnt(9)\n"
      "v_bitop3_b32 v171, v120, v96, 0 bitop3:0x10\n"
      "v_bitop3_b32 v170, v123, v98, 0 bitop3:0x14\n"
      "v_bitop3_b32 v174, v124, v107, 0 bitop3:0x14\n"
      "v_bitop3_b32 v168, v171, v122, v97 bitop3:0xd4\n"
      "v_bitop3_b32 v178, v131, v100, 0 bitop3:0x54\n"
      "v_bitop3_b32 v169, v104, v100, 0 bitop3:0x10\n"
      "v_bitop3_b32 v168, v168, v126, v101 bitop3:0xd4\n"
      "v_bitop3_b32 v173, v128, v131, 0 bitop3:0x40\n"
      "v_bitop3_b32 v171, v178, v128, v104 bitop3:0x10\n"
      "v_bitop3_b32 v168, v168, v121, v99 bitop3:0xd4\n"
      "v_bitop3_b32 v175, v173, v104, v100 bitop3:0xf8\n"
      "v_bitop3_b32 v172, v169, v128, v131 bitop3:0x40\n"
      "v_bitop3_b32 v179, v168, v123, v98 bitop3:0xd4\n"
      "v_bitop3_b32 v173, v169, v128, v131 bitop3:0xf4\n"
      "v_bitop3_b32 v182, v172, v175, v174 bitop3:0xec\n"
      "v_bitop3_b32 v168, v179, v130, v105 bitop3:0xd4\n"
      "v_bitop3_b32 v175, v169, v124, v107 bitop3:0xac\n"
      "v_bitop3_b32 v179, v124, v107, 0 bitop3:0x40\n"
      "v_bitop3_b32 v168, v168, v125, v102 bitop3:0xd4\n"
      "v_bitop3_b32 v168, v168, v129, v103 bitop3:0xd4\n"
      "v_bitop3_b32 v186, v168, v127, v106 bitop3:0xd4\n"
      "v_bitop3_b32 v168, v186, v131, v100 bitop3:0xd4\n"
      "v_bitop3_b32 v169, v168, v124, v107 bitop3:0xca\n"
      "v_bitop3_b32 v186, v168, v130, v105 bitop3:0xca\n"
      "v_bitop3_b32 v183, v168, v130, v105 bitop3:0xac\n"
      "v_bitop3_b32 v172, v168, v123, v98 bitop3:0x24\n"
      "v_bitop3_b32 v176, v168, v123, v98 bitop3:0xca\n"
      "v_bitop3_b32 v190, v168, v125, v102 bitop3:0xca\n"
      "v_bitop3_b32 v180, v168, v125, v102 bitop3:0xac\n"
      "v_bitop3_b32 v177, v172, v183, v186 bitop3:0xd4\n"
      "v_bitop3_b32 v194, v172, v183, v186 bitop3:0x96\n"
      "v_bitop3_b32 v172, v168, v129, v103 bitop3:0xca\n"
      "v_bitop3_b32 v198, v168, v129, v103 bitop3:0xac\n"
      "v_bitop3_b32 v181, v177, v180, v190 bitop3:0xd4\n"
      "v_bitop3_b32 v183, v177, v180, v190 bitop3:0x96\n"
      "v_bitop3_b32 v187, v168, v127, v106 bitop3:0xca\n"
      "v_bitop3_b32 v202, v168, v127, v106 bitop3:0xac\n"
      "v_bitop3_b32 v180, v181, v198, v172 bitop3:0xd4\n"
      "v_bitop3_b32 v198, v181, v198, v172 bitop3:0x96\n"
      "v_bitop3_b32 v206, v168, v120, v96 bitop3:0xac\n"
      "v_bitop3_b32 v180, v180, v202, v187 bitop3:0x96\n"
      "v_bitop3_b32 v202, v168, v120, v96 bitop3:0xca\n"
      "v_bitop3_b32 v210, v168, v122, v97 bitop3:0xac\n"
      "v_bitop3_b32 v177, v180, v198, 0 bitop3:0x54\n"
      "v_bitop3_b32 v198, v168, v122, v97 bitop3:0xca\n"
      "v_bitop3_b32 v214, v168, v126, v101 bitop3:0xac\n"
      "v_bitop3_b32 v218, v168, v126, v101 bitop3:0xca\n"
      "v_bitop3_b32 v181, v168, v121, v99 bitop3:0xac\n"
      "v_bitop3_b32 v222, v168, v121, v99 bitop3:0xca\n"
      "v_bitop3_b32 v168, v177, v131, v100 bitop3:0x08\n"
      "v_bitop3_b32 v177, v177, v131, v100 bitop3:0x80\n"
      "v_bitop3_b32 v185, v168, v206, 0 bitop3:0x40\n"
      "v_bitop3_b32 v191, v168, v210, 0 bitop3:0x40\n"
      "v_bitop3_b32 v180, v168, v214, 0 bitop3:0x40\n"
      "v_bitop3_b32 v195, v168, v181, 0 bitop3:0x40\n"
      "v_bitop3_b32 v199, v168, v170, v181 bitop3:0xe0\n"
      "v_bitop3_b32 v203, v168, v170, 0 bitop3:0x10\n"
      "v_bitop3_b32 v168, v195, v180, v170 bitop3:0xe4\n"
      "v_bitop3_b32 v180, v180, v191, v170 bitop3:0xe4\n"
      "v_bitop3_b32 v181, v191, v185, v170 bitop3:0xe4\n"
      "v_bitop3_b32 v191, v185, v170, 0 bitop3:0x40\n"
      "v_bitop3_b32 v185, v199, v180, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v184, v199, v194, 0 bitop3:0x10\n"
      "v_bitop3_b32 v189, v180, v191, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v170, v191, v177, v194 bitop3:0xec\n"
      "v_bitop3_b32 v206, v181, v194, 0 bitop3:0x40\n"
      "v_bitop3_b32 v180, v168, v181, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v177, v203, v168, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v181, v203, v194, 0 bitop3:0x10\n"
      "v_bitop3_b32 v194, v180, v189, v206 bitop3:0xfe\n"
      "v_bitop3_b32 v193, v177, v206, v183 bitop3:0xe4\n"
      "v_bitop3_b32 v191, v184, v189, v183 bitop3:0xe4\n"
      "v_bitop3_b32 v189, v194, v185, v183 bitop3:0xa8\n"
      "v_bitop3_b32 v195, v193, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v168, v181, v180, v183 bitop3:0xe4\n"
      "v_bitop3_b32 v199, v189, v170, 0 bitop3:0x54\n"
      "v_bitop3_b32 v189, v191, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v191, v168, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v185, v185, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v168, v177, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v203, v184, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v177, v181, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v170, v199, v174, 0 bitop3:0x04\n"
      "v_bitop3_b32 v180, v195, v170, 0 bitop3:0x40\n"
      "v_bitop3_b32 v181, v195, v170, 0 bitop3:0x14\n"
      "v_bitop3_b32 v193, v189, v180, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v189, v180, 0 bitop3:0x14\n"
      "v_bitop3_b32 v180, v191, v193, v202 bitop3:0xe8\n"
      "v_bitop3_b32 v191, v191, v193, v202 bitop3:0x96\n"
      "v_bitop3_b32 v195, v185, v180, v198 bitop3:0xe8\n"
      "v_bitop3_b32 v185, v185, v180, v198 bitop3:0x96\n"
      "v_bitop3_b32 v189, v168, v195, v218 bitop3:0xe8\n"
      "v_bitop3_b32 v195, v168, v195, v218 bitop3:0x96\n"
      "v_bitop3_b32 v207, v203, v189, v222 bitop3:0xe8\n"
      "v_bitop3_b32 v189, v203, v189, v222 bitop3:0x96\n"
      "v_bitop3_b32 v170, v177, v207, v174 bitop3:0x54\n"
      "v_bitop3_b32 v168, v177, v207, 0 bitop3:0x14\n"
      "v_bitop3_b32 v203, v168, v189, v195 bitop3:0x10\n"
      "v_bitop3_b32 v174, v203, v170, 0 bitop3:0x10\n"
      "v_bitop3_b32 v177, v203, v170, v185 bitop3:0xec\n"
      "v_bitop3_b32 v203, v174, v168, v191 bitop3:0x5c\n"
      "v_bitop3_b32 v168, v174, v191, 0 bitop3:0x04\n"
      "v_bitop3_b32 v185, v174, v185, v199 bitop3:0xac\n"
      "v_bitop3_b32 v180, v174, v199, 0 bitop3:0x04\n"
      "v_bitop3_b32 v170, v174, v189, v183 bitop3:0xac\n"
      "v_bitop3_b32 v194, v174, v183, 0 bitop3:0x04\n"
      "v_bitop3_b32 v198, v174, v195, v181 bitop3:0xac\n"
      "v_bitop3_b32 v202, v174, v181, 0 bitop3:0x04\n"
      "v_bitop3_b32 v183, v177, v203, 0 bitop3:0x04\n"
      "v_bitop3_b32 v206, v177, v203, v170 bitop3:0xf8\n"
      "v_bitop3_b32 v177, v177, v203, v198 bitop3:0xc4\n"
      "v_bitop3_b32 v191, v183, v198, v168 bitop3:0xac\n"
      "v_bitop3_b32 v168, v183, v168, v202 bitop3:0xac\n"
      "v_bitop3_b32 v184, v183, v170, v185 bitop3:0xac\n"
      "v_bitop3_b32 v181, v183, v185, v194 bitop3:0xac\n"
      "v_bitop3_b32 v195, v183, v194, v180 bitop3:0xac\n"
      "v_bitop3_b32 v199, v183, v180, 0 bitop3:0x04\n"
      "v_bitop3_b32 v185, v183, v202, 0 bitop3:0x04\n"
      "v_bitop3_b32 v170, v206, v168, v195 bitop3:0xca\n"
      "v_bitop3_b32 v203, v206, v181, v168 bitop3:0xca\n"
      "v_bitop3_b32 v194, v206, v191, v181 bitop3:0xca\n"
      "v_bitop3_b32 v168, v206, v184, v191 bitop3:0xca\n"
      "v_bitop3_b32 v198, v206, v177, v184 bitop3:0x3a\n"
      "v_bitop3_b32 v202, v206, v177, 0 bitop3:0x04\n"
      "v_bitop3_b32 v177, v206, v195, v185 bitop3:0xca\n"
      "v_bitop3_b32 v180, v206, v185, v199 bitop3:0xca\n"
      "v_bitop3_b32 v210, v206, v199, 0 bitop3:0x40\n"
      "v_bitop3_b32 v181, v171, v202, 0 bitop3:0x10\n"
      "v_bitop3_b32 v169, v202, v169, 0 bitop3:0x04\n"
      "v_bitop3_b32 v180, v177, v180, v210 bitop3:0xfe\n"
      "v_bitop3_b32 v171, v203, v170, 0 bitop3:0x40\n"
      "v_bitop3_b32 v178, v169, v179, v178 bitop3:0xe4\n"
      "v_bitop3_b32 v108, v180, v203, v170 bitop3:0x64\n"
      "v_bitop3_b32 v169, v171, v194, 0 bitop3:0x40\n"
      "v_bitop3_b32 v109, v171, v194, 0 bitop3:0x14\n"
      "v_bitop3_b32 v119, v175, v178, v173 bitop3:0xe4\n"
      "v_bitop3_b32 v171, v169, v168, 0 bitop3:0x40\n"
      "v_bitop3_b32 v113, v169, v168, 0 bitop3:0x14\n"
      "v_bitop3_b32 v175, v183, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v170, v183, v174, 0 bitop3:0x54\n"
      "v_bitop3_b32 v169, v171, v198, 0 bitop3:0x40\n"
      "v_bitop3_b32 v111, v171, v198, 0 bitop3:0x14\n"
      "v_bitop3_b32 v168, v169, v206, v176 bitop3:0xe8\n"
      "v_bitop3_b32 v110, v169, v206, v176 bitop3:0x96\n"
      "v_bitop3_b32 v176, v168, v183, v186 bitop3:0xe8\n"
      "v_bitop3_b32 v117, v168, v183, v186 bitop3:0x96\n"
      "v_bitop3_b32 v169, v176, v175, v190 bitop3:0xe8\n"
      "v_bitop3_b32 v114, v176, v175, v190 bitop3:0x96\n"
      "v_bitop3_b32 v168, v169, v170, v172 bitop3:0xe8\n"
      "v_bitop3_b32 v115, v169, v170, v172 bitop3:0x96\n"
      "v_bitop3_b32 v171, v168, v170, v187 bitop3:0xe8\n"
      "v_bitop3_b32 v118, v168, v170, v187 bitop3:0x96\n"
      "v_bitop3_b32 v168, v171, v170, 0 bitop3:0x14\n"
      "v_bitop3_b32 v171, v181, v171, v170 bitop3:0x40\n"
      "v_bitop3_b32 v116, v171, v173, v182 bitop3:0xfe\n"
      "v_bitop3_b32 v112, v181, v182, v168 bitop3:0xdc\n"
      "s_waitcnt lgkmcnt(6)\n"
      "v_bitop3_b32 v171, v132, v108, 0 bitop3:0x10\n"
      "v_bitop3_b32 v170, v135, v110, 0 bitop3:0x14\n"
      "v_bitop3_b32 v174, v136, v119, 0 bitop3:0x14\n"
      "v_bitop3_b32 v168, v171, v134, v109 bitop3:0xd4\n"
      "v_bitop3_b32 v178, v143, v112, 0 bitop3:0x54\n"
      "v_bitop3_b32 v169, v116, v112, 0 bitop3:0x10\n"
      "v_bitop3_b32 v168, v168, v138, v113 bitop3:0xd4\n"
      "v_bitop3_b32 v173, v140, v143, 0 bitop3:0x40\n"
      "v_bitop3_b32 v171, v178, v140, v116 bitop3:0x10\n"
      "v_bitop3_b32 v168, v168, v133, v111 bitop3:0xd4\n"
      "v_bitop3_b32 v175, v173, v116, v112 bitop3:0xf8\n"
      "v_bitop3_b32 v172, v169, v140, v143 bitop3:0x40\n"
      "v_bitop3_b32 v179, v168, v135, v110 bitop3:0xd4\n"
      "v_bitop3_b32 v173, v169, v140, v143 bitop3:0xf4\n"
      "v_bitop3_b32 v182, v172, v175, v174 bitop3:0xec\n"
      "v_bitop3_b32 v168, v179, v142, v117 bitop3:0xd4\n"
      "v_bitop3_b32 v175, v169, v136, v119 bitop3:0xac\n"
      "v_bitop3_b32 v179, v136, v119, 0 bitop3:0x40\n"
      "v_bitop3_b32 v168, v168, v137, v114 bitop3:0xd4\n"
      "v_bitop3_b32 v168, v168, v141, v115 bitop3:0xd4\n"
      "v_bitop3_b32 v186, v168, v139, v118 bitop3:0xd4\n"
      "v_bitop3_b32 v168, v186, v143, v112 bitop3:0xd4\n"
      "v_bitop3_b32 v169, v168, v136, v119 bitop3:0xca\n"
      "v_bitop3_b32 v186, v168, v142, v117 bitop3:0xca\n"
      "v_bitop3_b32 v183, v168, v142, v117 bitop3:0xac\n"
      "v_bitop3_b32 v172, v168, v135, v110 bitop3:0x24\n"
      "v_bitop3_b32 v176, v168, v135, v110 bitop3:0xca\n"
      "v_bitop3_b32 v190, v168, v137, v114 bitop3:0xca\n"
      "v_bitop3_b32 v180, v168, v137, v114 bitop3:0xac\n"
      "v_bitop3_b32 v177, v172, v183, v186 bitop3:0xd4\n"
      "v_bitop3_b32 v194, v172, v183, v186 bitop3:0x96\n"
      "v_bitop3_b32 v172, v168, v141, v115 bitop3:0xca\n"
      "v_bitop3_b32 v198, v168, v141, v115 bitop3:0xac\n"
      "v_bitop3_b32 v181, v177, v180, v190 bitop3:0xd4\n"
      "v_bitop3_b32 v183, v177, v180, v190 bitop3:0x96\n"
      "v_bitop3_b32 v187, v168, v139, v118 bitop3:0xca\n"
      "v_bitop3_b32 v202, v168, v139, v118 bitop3:0xac\n"
      "v_bitop3_b32 v180, v181, v198, v172 bitop3:0xd4\n"
      "v_bitop3_b32 v198, v181, v198, v172 bitop3:0x96\n"
      "v_bitop3_b32 v206, v168, v132, v108 bitop3:0xac\n"
      "v_bitop3_b32 v180, v180, v202, v187 bitop3:0x96\n"
      "v_bitop3_b32 v202, v168, v132, v108 bitop3:0xca\n"
      "v_bitop3_b32 v210, v168, v134, v109 bitop3:0xac\n"
      "v_bitop3_b32 v177, v180, v198, 0 bitop3:0x54\n"
      "v_bitop3_b32 v198, v168, v134, v109 bitop3:0xca\n"
      "v_bitop3_b32 v214, v168, v138, v113 bitop3:0xac\n"
      "v_bitop3_b32 v218, v168, v138, v113 bitop3:0xca\n"
      "v_bitop3_b32 v181, v168, v133, v111 bitop3:0xac\n"
      "v_bitop3_b32 v222, v168, v133, v111 bitop3:0xca\n"
      "v_bitop3_b32 v168, v177, v143, v112 bitop3:0x08\n"
      "v_bitop3_b32 v177, v177, v143, v112 bitop3:0x80\n"
      "v_bitop3_b32 v185, v168, v206, 0 bitop3:0x40\n"
      "v_bitop3_b32 v191, v168, v210, 0 bitop3:0x40\n"
      "v_bitop3_b32 v180, v168, v214, 0 bitop3:0x40\n"
      "v_bitop3_b32 v195, v168, v181, 0 bitop3:0x40\n"
      "v_bitop3_b32 v199, v168, v170, v181 bitop3:0xe0\n"
      "v_bitop3_b32 v203, v168, v170, 0 bitop3:0x10\n"
      "v_bitop3_b32 v168, v195, v180, v170 bitop3:0xe4\n"
      "v_bitop3_b32 v180, v180, v191, v170 bitop3:0xe4\n"
      "v_bitop3_b32 v181, v191, v185, v170 bitop3:0xe4\n"
      "v_bitop3_b32 v191, v185, v170, 0 bitop3:0x40\n"
      "v_bitop3_b32 v185, v199, v180, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v184, v199, v194, 0 bitop3:0x10\n"
      "v_bitop3_b32 v189, v180, v191, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v170, v191, v177, v194 bitop3:0xec\n"
      "v_bitop3_b32 v206, v181, v194, 0 bitop3:0x40\n"
      "v_bitop3_b32 v180, v168, v181, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v177, v203, v168, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v181, v203, v194, 0 bitop3:0x10\n"
      "v_bitop3_b32 v194, v180, v189, v206 bitop3:0xfe\n"
      "v_bitop3_b32 v193, v177, v206, v183 bitop3:0xe4\n"
      "v_bitop3_b32 v191, v184, v189, v183 bitop3:0xe4\n"
      "v_bitop3_b32 v189, v194, v185, v183 bitop3:0xa8\n"
      "v_bitop3_b32 v195, v193, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v168, v181, v180, v183 bitop3:0xe4\n"
      "v_bitop3_b32 v199, v189, v170, 0 bitop3:0x54\n"
      "v_bitop3_b32 v189, v191, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v191, v168, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v185, v185, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v168, v177, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v203, v184, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v177, v181, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v170, v199, v174, 0 bitop3:0x04\n"
      "v_bitop3_b32 v180, v195, v170, 0 bitop3:0x40\n"
      "v_bitop3_b32 v181, v195, v170, 0 bitop3:0x14\n"
      "v_bitop3_b32 v193, v189, v180, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v189, v180, 0 bitop3:0x14\n"
      "v_bitop3_b32 v180, v191, v193, v202 bitop3:0xe8\n"
      "v_bitop3_b32 v191, v191, v193, v202 bitop3:0x96\n"
      "v_bitop3_b32 v195, v185, v180, v198 bitop3:0xe8\n"
      "v_bitop3_b32 v185, v185, v180, v198 bitop3:0x96\n"
      "v_bitop3_b32 v189, v168, v195, v218 bitop3:0xe8\n"
      "v_bitop3_b32 v195, v168, v195, v218 bitop3:0x96\n"
      "v_bitop3_b32 v207, v203, v189, v222 bitop3:0xe8\n"
      "v_bitop3_b32 v189, v203, v189, v222 bitop3:0x96\n"
      "v_bitop3_b32 v170, v177, v207, v174 bitop3:0x54\n"
      "v_bitop3_b32 v168, v177, v207, 0 bitop3:0x14\n"
      "v_bitop3_b32 v203, v168, v189, v195 bitop3:0x10\n"
      "v_bitop3_b32 v174, v203, v170, 0 bitop3:0x10\n"
      "v_bitop3_b32 v177, v203, v170, v185 bitop3:0xec\n"
      "v_bitop3_b32 v203, v174, v168, v191 bitop3:0x5c\n"
      "v_bitop3_b32 v168, v174, v191, 0 bitop3:0x04\n"
      "v_bitop3_b32 v185, v174, v185, v199 bitop3:0xac\n"
      "v_bitop3_b32 v180, v174, v199, 0 bitop3:0x04\n"
      "v_bitop3_b32 v170, v174, v189, v183 bitop3:0xac\n"
      "v_bitop3_b32 v194, v174, v183, 0 bitop3:0x04\n"
      "v_bitop3_b32 v198, v174, v195, v181 bitop3:0xac\n"
      "v_bitop3_b32 v202, v174, v181, 0 bitop3:0x04\n"
      "v_bitop3_b32 v183, v177, v203, 0 bitop3:0x04\n"
      "v_bitop3_b32 v206, v177, v203, v170 bitop3:0xf8\n"
      "v_bitop3_b32 v177, v177, v203, v198 bitop3:0xc4\n"
      "v_bitop3_b32 v191, v183, v198, v168 bitop3:0xac\n"
      "v_bitop3_b32 v168, v183, v168, v202 bitop3:0xac\n"
      "v_bitop3_b32 v184, v183, v170, v185 bitop3:0xac\n"
      "v_bitop3_b32 v181, v183, v185, v194 bitop3:0xac\n"
      "v_bitop3_b32 v195, v183, v194, v180 bitop3:0xac\n"
      "v_bitop3_b32 v199, v183, v180, 0 bitop3:0x04\n"
      "v_bitop3_b32 v185, v183, v202, 0 bitop3:0x04\n"
      "v_bitop3_b32 v170, v206, v168, v195 bitop3:0xca\n"
      "v_bitop3_b32 v203, v206, v181, v168 bitop3:0xca\n"
      "v_bitop3_b32 v194, v206, v191, v181 bitop3:0xca\n"
      "v_bitop3_b32 v168, v206, v184, v191 bitop3:0xca\n"
      "v_bitop3_b32 v198, v206, v177, v184 bitop3:0x3a\n"
      "v_bitop3_b32 v202, v206, v177, 0 bitop3:0x04\n"
      "v_bitop3_b32 v177, v206, v195, v185 bitop3:0xca\n"
      "v_bitop3_b32 v180, v206, v185, v199 bitop3:0xca\n"
      "v_bitop3_b32 v210, v206, v199, 0 bitop3:0x40\n"
      "v_bitop3_b32 v181, v171, v202, 0 bitop3:0x10\n"
      "v_bitop3_b32 v169, v202, v169, 0 bitop3:0x04\n"
      "v_bitop3_b32 v180, v177, v180, v210 bitop3:0xfe\n"
      "v_bitop3_b32 v171, v203, v170, 0 bitop3:0x40\n"
      "v_bitop3_b32 v178, v169, v179, v178 bitop3:0xe4\n"
      "v_bitop3_b32 v96, v180, v203, v170 bitop3:0x64\n"
      "v_bitop3_b32 v169, v171, v194, 0 bitop3:0x40\n"
      "v_bitop3_b32 v97, v171, v194, 0 bitop3:0x14\n"
      "v_bitop3_b32 v107, v175, v178, v173 bitop3:0xe4\n"
      "v_bitop3_b32 v171, v169, v168, 0 bitop3:0x40\n"
      "v_bitop3_b32 v101, v169, v168, 0 bitop3:0x14\n"
      "v_bitop3_b32 v175, v183, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v170, v183, v174, 0 bitop3:0x54\n"
      "v_bitop3_b32 v169, v171, v198, 0 bitop3:0x40\n"
      "v_bitop3_b32 v99, v171, v198, 0 bitop3:0x14\n"
      "v_bitop3_b32 v168, v169, v206, v176 bitop3:0xe8\n"
      "v_bitop3_b32 v98, v169, v206, v176 bitop3:0x96\n"
      "v_bitop3_b32 v176, v168, v183, v186 bitop3:0xe8\n"
      "v_bitop3_b32 v105, v168, v183, v186 bitop3:0x96\n"
      "v_bitop3_b32 v169, v176, v175, v190 bitop3:0xe8\n"
      "v_bitop3_b32 v102, v176, v175, v190 bitop3:0x96\n"
      "v_bitop3_b32 v168, v169, v170, v172 bitop3:0xe8\n"
      "v_bitop3_b32 v103, v169, v170, v172 bitop3:0x96\n"
      "v_bitop3_b32 v171, v168, v170, v187 bitop3:0xe8\n"
      "v_bitop3_b32 v106, v168, v170, v187 bitop3:0x96\n"
      "v_bitop3_b32 v168, v171, v170, 0 bitop3:0x14\n"
      "v_bitop3_b32 v171, v181, v171, v170 bitop3:0x40\n"
      "v_bitop3_b32 v104, v171, v173, v182 bitop3:0xfe\n"
      "v_bitop3_b32 v100, v181, v182, v168 bitop3:0xdc\n"
      "s_waitcnt lgkmcnt(3)\n"
      "v_bitop3_b32 v171, v144, v96, 0 bitop3:0x10\n"
      "v_bitop3_b32 v170, v147, v98, 0 bitop3:0x14\n"
      "v_bitop3_b32 v174, v148, v107, 0 bitop3:0x14\n"
      "v_bitop3_b32 v168, v171, v146, v97 bitop3:0xd4\n"
      "v_bitop3_b32 v178, v155, v100, 0 bitop3:0x54\n"
      "v_bitop3_b32 v169, v104, v100, 0 bitop3:0x10\n"
      "v_bitop3_b32 v168, v168, v150, v101 bitop3:0xd4\n"
      "v_bitop3_b32 v173, v152, v155, 0 bitop3:0x40\n"
      "v_bitop3_b32 v171, v178, v152, v104 bitop3:0x10\n"
      "v_bitop3_b32 v168, v168, v145, v99 bitop3:0xd4\n"
      "v_bitop3_b32 v175, v173, v104, v100 bitop3:0xf8\n"
      "v_bitop3_b32 v172, v169, v152, v155 bitop3:0x40\n"
      "v_bitop3_b32 v179, v168, v147, v98 bitop3:0xd4\n"
      "v_bitop3_b32 v173, v169, v152, v155 bitop3:0xf4\n"
      "v_bitop3_b32 v182, v172, v175, v174 bitop3:0xec\n"
      "v_bitop3_b32 v168, v179, v154, v105 bitop3:0xd4\n"
      "v_bitop3_b32 v175, v169, v148, v107 bitop3:0xac\n"
      "v_bitop3_b32 v179, v148, v107, 0 bitop3:0x40\n"
      "v_bitop3_b32 v168, v168, v149, v102 bitop3:0xd4\n"
      "v_bitop3_b32 v168, v168, v153, v103 bitop3:0xd4\n"
      "v_bitop3_b32 v186, v168, v151, v106 bitop3:0xd4\n"
      "v_bitop3_b32 v168, v186, v155, v100 bitop3:0xd4\n"
      "v_bitop3_b32 v169, v168, v148, v107 bitop3:0xca\n"
      "v_bitop3_b32 v186, v168, v154, v105 bitop3:0xca\n"
      "v_bitop3_b32 v183, v168, v154, v105 bitop3:0xac\n"
      "v_bitop3_b32 v172, v168, v147, v98 bitop3:0x24\n"
      "v_bitop3_b32 v176, v168, v147, v98 bitop3:0xca\n"
      "v_bitop3_b32 v190, v168, v149, v102 bitop3:0xca\n"
      "v_bitop3_b32 v180, v168, v149, v102 bitop3:0xac\n"
      "v_bitop3_b32 v177, v172, v183, v186 bitop3:0xd4\n"
      "v_bitop3_b32 v194, v172, v183, v186 bitop3:0x96\n"
      "v_bitop3_b32 v172, v168, v153, v103 bitop3:0xca\n"
      "v_bitop3_b32 v198, v168, v153, v103 bitop3:0xac\n"
      "v_bitop3_b32 v181, v177, v180, v190 bitop3:0xd4\n"
      "v_bitop3_b32 v183, v177, v180, v190 bitop3:0x96\n"
      "v_bitop3_b32 v187, v168, v151, v106 bitop3:0xca\n"
      "v_bitop3_b32 v202, v168, v151, v106 bitop3:0xac\n"
      "v_bitop3_b32 v180, v181, v198, v172 bitop3:0xd4\n"
      "v_bitop3_b32 v198, v181, v198, v172 bitop3:0x96\n"
      "v_bitop3_b32 v206, v168, v144, v96 bitop3:0xac\n"
      "v_bitop3_b32 v180, v180, v202, v187 bitop3:0x96\n"
      "v_bitop3_b32 v202, v168, v144, v96 bitop3:0xca\n"
      "v_bitop3_b32 v210, v168, v146, v97 bitop3:0xac\n"
      "v_bitop3_b32 v177, v180, v198, 0 bitop3:0x54\n"
      "v_bitop3_b32 v198, v168, v146, v97 bitop3:0xca\n"
      "v_bitop3_b32 v214, v168, v150, v101 bitop3:0xac\n"
      "v_bitop3_b32 v218, v168, v150, v101 bitop3:0xca\n"
      "v_bitop3_b32 v181, v168, v145, v99 bitop3:0xac\n"
      "v_bitop3_b32 v222, v168, v145, v99 bitop3:0xca\n"
      "v_bitop3_b32 v168, v177, v155, v100 bitop3:0x08\n"
      "v_bitop3_b32 v177, v177, v155, v100 bitop3:0x80\n"
      "v_bitop3_b32 v185, v168, v206, 0 bitop3:0x40\n"
      "v_bitop3_b32 v191, v168, v210, 0 bitop3:0x40\n"
      "v_bitop3_b32 v180, v168, v214, 0 bitop3:0x40\n"
      "v_bitop3_b32 v195, v168, v181, 0 bitop3:0x40\n"
      "v_bitop3_b32 v199, v168, v170, v181 bitop3:0xe0\n"
      "v_bitop3_b32 v203, v168, v170, 0 bitop3:0x10\n"
      "v_bitop3_b32 v168, v195, v180, v170 bitop3:0xe4\n"
      "v_bitop3_b32 v180, v180, v191, v170 bitop3:0xe4\n"
      "v_bitop3_b32 v181, v191, v185, v170 bitop3:0xe4\n"
      "v_bitop3_b32 v191, v185, v170, 0 bitop3:0x40\n"
      "v_bitop3_b32 v185, v199, v180, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v184, v199, v194, 0 bitop3:0x10\n"
      "v_bitop3_b32 v189, v180, v191, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v170, v191, v177, v194 bitop3:0xec\n"
      "v_bitop3_b32 v206, v181, v194, 0 bitop3:0x40\n"
      "v_bitop3_b32 v180, v168, v181, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v177, v203, v168, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v181, v203, v194, 0 bitop3:0x10\n"
      "v_bitop3_b32 v194, v180, v189, v206 bitop3:0xfe\n"
      "v_bitop3_b32 v193, v177, v206, v183 bitop3:0xe4\n"
      "v_bitop3_b32 v191, v184, v189, v183 bitop3:0xe4\n"
      "v_bitop3_b32 v189, v194, v185, v183 bitop3:0xa8\n"
      "v_bitop3_b32 v195, v193, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v168, v181, v180, v183 bitop3:0xe4\n"
      "v_bitop3_b32 v199, v189, v170, 0 bitop3:0x54\n"
      "v_bitop3_b32 v189, v191, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v191, v168, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v185, v185, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v168, v177, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v203, v184, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v177, v181, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v170, v199, v174, 0 bitop3:0x04\n"
      "v_bitop3_b32 v180, v195, v170, 0 bitop3:0x40\n"
      "v_bitop3_b32 v181, v195, v170, 0 bitop3:0x14\n"
      "v_bitop3_b32 v193, v189, v180, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v189, v180, 0 bitop3:0x14\n"
      "v_bitop3_b32 v180, v191, v193, v202 bitop3:0xe8\n"
      "v_bitop3_b32 v191, v191, v193, v202 bitop3:0x96\n"
      "v_bitop3_b32 v195, v185, v180, v198 bitop3:0xe8\n"
      "v_bitop3_b32 v185, v185, v180, v198 bitop3:0x96\n"
      "v_bitop3_b32 v189, v168, v195, v218 bitop3:0xe8\n"
      "v_bitop3_b32 v195, v168, v195, v218 bitop3:0x96\n"
      "v_bitop3_b32 v207, v203, v189, v222 bitop3:0xe8\n"
      "v_bitop3_b32 v189, v203, v189, v222 bitop3:0x96\n"
      "v_bitop3_b32 v170, v177, v207, v174 bitop3:0x54\n"
      "v_bitop3_b32 v168, v177, v207, 0 bitop3:0x14\n"
      "v_bitop3_b32 v203, v168, v189, v195 bitop3:0x10\n"
      "v_bitop3_b32 v174, v203, v170, 0 bitop3:0x10\n"
      "v_bitop3_b32 v177, v203, v170, v185 bitop3:0xec\n"
      "v_bitop3_b32 v203, v174, v168, v191 bitop3:0x5c\n"
      "v_bitop3_b32 v168, v174, v191, 0 bitop3:0x04\n"
      "v_bitop3_b32 v185, v174, v185, v199 bitop3:0xac\n"
      "v_bitop3_b32 v180, v174, v199, 0 bitop3:0x04\n"
      "v_bitop3_b32 v170, v174, v189, v183 bitop3:0xac\n"
      "v_bitop3_b32 v194, v174, v183, 0 bitop3:0x04\n"
      "v_bitop3_b32 v198, v174, v195, v181 bitop3:0xac\n"
      "v_bitop3_b32 v202, v174, v181, 0 bitop3:0x04\n"
      "v_bitop3_b32 v183, v177, v203, 0 bitop3:0x04\n"
      "v_bitop3_b32 v206, v177, v203, v170 bitop3:0xf8\n"
      "v_bitop3_b32 v177, v177, v203, v198 bitop3:0xc4\n"
      "v_bitop3_b32 v191, v183, v198, v168 bitop3:0xac\n"
      "v_bitop3_b32 v168, v183, v168, v202 bitop3:0xac\n"
      "v_bitop3_b32 v184, v183, v170, v185 bitop3:0xac\n"
      "v_bitop3_b32 v181, v183, v185, v194 bitop3:0xac\n"
      "v_bitop3_b32 v195, v183, v194, v180 bitop3:0xac\n"
      "v_bitop3_b32 v199, v183, v180, 0 bitop3:0x04\n"
      "v_bitop3_b32 v185, v183, v202, 0 bitop3:0x04\n"
      "v_bitop3_b32 v170, v206, v168, v195 bitop3:0xca\n"
      "v_bitop3_b32 v203, v206, v181, v168 bitop3:0xca\n"
      "v_bitop3_b32 v194, v206, v191, v181 bitop3:0xca\n"
      "v_bitop3_b32 v168, v206, v184, v191 bitop3:0xca\n"
      "v_bitop3_b32 v198, v206, v177, v184 bitop3:0x3a\n"
      "v_bitop3_b32 v202, v206, v177, 0 bitop3:0x04\n"
      "v_bitop3_b32 v177, v206, v195, v185 bitop3:0xca\n"
      "v_bitop3_b32 v180, v206, v185, v199 bitop3:0xca\n"
      "v_bitop3_b32 v210, v206, v199, 0 bitop3:0x40\n"
      "v_bitop3_b32 v181, v171, v202, 0 bitop3:0x10\n"
      "v_bitop3_b32 v169, v202, v169, 0 bitop3:0x04\n"
      "v_bitop3_b32 v180, v177, v180, v210 bitop3:0xfe\n"
      "v_bitop3_b32 v171, v203, v170, 0 bitop3:0x40\n"
      "v_bitop3_b32 v178, v169, v179, v178 bitop3:0xe4\n"
      "v_bitop3_b32 v108, v180, v203, v170 bitop3:0x64\n"
      "v_bitop3_b32 v169, v171, v194, 0 bitop3:0x40\n"
      "v_bitop3_b32 v109, v171, v194, 0 bitop3:0x14\n"
      "v_bitop3_b32 v119, v175, v178, v173 bitop3:0xe4\n"
      "v_bitop3_b32 v171, v169, v168, 0 bitop3:0x40\n"
      "v_bitop3_b32 v113, v169, v168, 0 bitop3:0x14\n"
      "v_bitop3_b32 v175, v183, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v170, v183, v174, 0 bitop3:0x54\n"
      "v_bitop3_b32 v169, v171, v198, 0 bitop3:0x40\n"
      "v_bitop3_b32 v111, v171, v198, 0 bitop3:0x14\n"
      "v_bitop3_b32 v168, v169, v206, v176 bitop3:0xe8\n"
      "v_bitop3_b32 v110, v169, v206, v176 bitop3:0x96\n"
      "v_bitop3_b32 v176, v168, v183, v186 bitop3:0xe8\n"
      "v_bitop3_b32 v117, v168, v183, v186 bitop3:0x96\n"
      "v_bitop3_b32 v169, v176, v175, v190 bitop3:0xe8\n"
      "v_bitop3_b32 v114, v176, v175, v190 bitop3:0x96\n"
      "v_bitop3_b32 v168, v169, v170, v172 bitop3:0xe8\n"
      "v_bitop3_b32 v115, v169, v170, v172 bitop3:0x96\n"
      "v_bitop3_b32 v171, v168, v170, v187 bitop3:0xe8\n"
      "v_bitop3_b32 v118, v168, v170, v187 bitop3:0x96\n"
      "v_bitop3_b32 v168, v171, v170, 0 bitop3:0x14\n"
      "v_bitop3_b32 v171, v181, v171, v170 bitop3:0x40\n"
      "v_bitop3_b32 v116, v171, v173, v182 bitop3:0xfe\n"
      "v_bitop3_b32 v112, v181, v182, v168 bitop3:0xdc\n"
      "s_waitcnt lgkmcnt(0)\n"
      "v_bitop3_b32 v171, v156, v108, 0 bitop3:0x10\n"
      "v_bitop3_b32 v170, v159, v110, 0 bitop3:0x14\n"
      "v_bitop3_b32 v174, v160, v119, 0 bitop3:0x14\n"
      "v_bitop3_b32 v168, v171, v158, v109 bitop3:0xd4\n"
      "v_bitop3_b32 v178, v167, v112, 0 bitop3:0x54\n"
      "v_bitop3_b32 v169, v116, v112, 0 bitop3:0x10\n"
      "v_bitop3_b32 v168, v168, v162, v113 bitop3:0xd4\n"
      "v_bitop3_b32 v173, v164, v167, 0 bitop3:0x40\n"
      "v_bitop3_b32 v171, v178, v164, v116 bitop3:0x10\n"
      "v_bitop3_b32 v168, v168, v157, v111 bitop3:0xd4\n"
      "v_bitop3_b32 v175, v173, v116, v112 bitop3:0xf8\n"
      "v_bitop3_b32 v172, v169, v164, v167 bitop3:0x40\n"
      "v_bitop3_b32 v179, v168, v159, v110 bitop3:0xd4\n"
      "v_bitop3_b32 v173, v169, v164, v167 bitop3:0xf4\n"
      "v_bitop3_b32 v182, v172, v175, v174 bitop3:0xec\n"
      "v_bitop3_b32 v168, v179, v166, v117 bitop3:0xd4\n"
      "v_bitop3_b32 v175, v169, v160, v119 bitop3:0xac\n"
      "v_bitop3_b32 v179, v160, v119, 0 bitop3:0x40\n"
      "v_bitop3_b32 v168, v168, v161, v114 bitop3:0xd4\n"
      "v_bitop3_b32 v168, v168, v165, v115 bitop3:0xd4\n"
      "v_bitop3_b32 v186, v168, v163, v118 bitop3:0xd4\n"
      "v_bitop3_b32 v168, v186, v167, v112 bitop3:0xd4\n"
      "v_bitop3_b32 v169, v168, v160, v119 bitop3:0xca\n"
      "v_bitop3_b32 v186, v168, v166, v117 bitop3:0xca\n"
      "v_bitop3_b32 v183, v168, v166, v117 bitop3:0xac\n"
      "v_bitop3_b32 v172, v168, v159, v110 bitop3:0x24\n"
      "v_bitop3_b32 v176, v168, v159, v110 bitop3:0xca\n"
      "v_bitop3_b32 v190, v168, v161, v114 bitop3:0xca\n"
      "v_bitop3_b32 v180, v168, v161, v114 bitop3:0xac\n"
      "v_bitop3_b32 v177, v172, v183, v186 bitop3:0xd4\n"
      "v_bitop3_b32 v194, v172, v183, v186 bitop3:0x96\n"
      "v_bitop3_b32 v172, v168, v165, v115 bitop3:0xca\n"
      "v_bitop3_b32 v198, v168, v165, v115 bitop3:0xac\n"
      "v_bitop3_b32 v181, v177, v180, v190 bitop3:0xd4\n"
      "v_bitop3_b32 v183, v177, v180, v190 bitop3:0x96\n"
      "v_bitop3_b32 v187, v168, v163, v118 bitop3:0xca\n"
      "v_bitop3_b32 v202, v168, v163, v118 bitop3:0xac\n"
      "v_bitop3_b32 v180, v181, v198, v172 bitop3:0xd4\n"
      "v_bitop3_b32 v198, v181, v198, v172 bitop3:0x96\n"
      "v_bitop3_b32 v206, v168, v156, v108 bitop3:0xac\n"
      "v_bitop3_b32 v180, v180, v202, v187 bitop3:0x96\n"
      "v_bitop3_b32 v202, v168, v156, v108 bitop3:0xca\n"
      "v_bitop3_b32 v210, v168, v158, v109 bitop3:0xac\n"
      "v_bitop3_b32 v177, v180, v198, 0 bitop3:0x54\n"
      "v_bitop3_b32 v198, v168, v158, v109 bitop3:0xca\n"
      "v_bitop3_b32 v214, v168, v162, v113 bitop3:0xac\n"
      "v_bitop3_b32 v218, v168, v162, v113 bitop3:0xca\n"
      "v_bitop3_b32 v181, v168, v157, v111 bitop3:0xac\n"
      "v_bitop3_b32 v222, v168, v157, v111 bitop3:0xca\n"
      "v_bitop3_b32 v168, v177, v167, v112 bitop3:0x08\n"
      "v_bitop3_b32 v177, v177, v167, v112 bitop3:0x80\n"
      "v_bitop3_b32 v185, v168, v206, 0 bitop3:0x40\n"
      "v_bitop3_b32 v191, v168, v210, 0 bitop3:0x40\n"
      "v_bitop3_b32 v180, v168, v214, 0 bitop3:0x40\n"
      "v_bitop3_b32 v195, v168, v181, 0 bitop3:0x40\n"
      "v_bitop3_b32 v199, v168, v170, v181 bitop3:0xe0\n"
      "v_bitop3_b32 v203, v168, v170, 0 bitop3:0x10\n"
      "v_bitop3_b32 v168, v195, v180, v170 bitop3:0xe4\n"
      "v_bitop3_b32 v180, v180, v191, v170 bitop3:0xe4\n"
      "v_bitop3_b32 v181, v191, v185, v170 bitop3:0xe4\n"
      "v_bitop3_b32 v191, v185, v170, 0 bitop3:0x40\n"
      "v_bitop3_b32 v185, v199, v180, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v184, v199, v194, 0 bitop3:0x10\n"
      "v_bitop3_b32 v189, v180, v191, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v170, v191, v177, v194 bitop3:0xec\n"
      "v_bitop3_b32 v206, v181, v194, 0 bitop3:0x40\n"
      "v_bitop3_b32 v180, v168, v181, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v177, v203, v168, v194 bitop3:0xe4\n"
      "v_bitop3_b32 v181, v203, v194, 0 bitop3:0x10\n"
      "v_bitop3_b32 v194, v180, v189, v206 bitop3:0xfe\n"
      "v_bitop3_b32 v193, v177, v206, v183 bitop3:0xe4\n"
      "v_bitop3_b32 v191, v184, v189, v183 bitop3:0xe4\n"
      "v_bitop3_b32 v189, v194, v185, v183 bitop3:0xa8\n"
      "v_bitop3_b32 v195, v193, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v168, v181, v180, v183 bitop3:0xe4\n"
      "v_bitop3_b32 v199, v189, v170, 0 bitop3:0x54\n"
      "v_bitop3_b32 v189, v191, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v191, v168, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v185, v185, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v168, v177, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v203, v184, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v177, v181, v183, v174 bitop3:0x9a\n"
      "v_bitop3_b32 v170, v199, v174, 0 bitop3:0x04\n"
      "v_bitop3_b32 v180, v195, v170, 0 bitop3:0x40\n"
      "v_bitop3_b32 v181, v195, v170, 0 bitop3:0x14\n"
      "v_bitop3_b32 v193, v189, v180, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v189, v180, 0 bitop3:0x14\n"
      "v_bitop3_b32 v180, v191, v193, v202 bitop3:0xe8\n"
      "v_bitop3_b32 v191, v191, v193, v202 bitop3:0x96\n"
      "v_bitop3_b32 v195, v185, v180, v198 bitop3:0xe8\n"
      "v_bitop3_b32 v185, v185, v180, v198 bitop3:0x96\n"
      "v_bitop3_b32 v189, v168, v195, v218 bitop3:0xe8\n"
      "v_bitop3_b32 v195, v168, v195, v218 bitop3:0x96\n"
      "v_bitop3_b32 v207, v203, v189, v222 bitop3:0xe8\n"
      "v_bitop3_b32 v189, v203, v189, v222 bitop3:0x96\n"
      "v_bitop3_b32 v170, v177, v207, v174 bitop3:0x54\n"
      "v_bitop3_b32 v168, v177, v207, 0 bitop3:0x14\n"
      "v_bitop3_b32 v203, v168, v189, v195 bitop3:0x10\n"
      "v_bitop3_b32 v174, v203, v170, 0 bitop3:0x10\n"
      "v_bitop3_b32 v177, v203, v170, v185 bitop3:0xec\n"
      "v_bitop3_b32 v203, v174, v168, v191 bitop3:0x5c\n"
      "v_bitop3_b32 v168, v174, v191, 0 bitop3:0x04\n"
      "v_bitop3_b32 v185, v174, v185, v199 bitop3:0xac\n"
      "v_bitop3_b32 v180, v174, v199, 0 bitop3:0x04\n"
      "v_bitop3_b32 v170, v174, v189, v183 bitop3:0xac\n"
      "v_bitop3_b32 v194, v174, v183, 0 bitop3:0x04\n"
      "v_bitop3_b32 v198, v174, v195, v181 bitop3:0xac\n"
      "v_bitop3_b32 v202, v174, v181, 0 bitop3:0x04\n"
      "v_bitop3_b32 v183, v177, v203, 0 bitop3:0x04\n"
      "v_bitop3_b32 v206, v177, v203, v170 bitop3:0xf8\n"
      "v_bitop3_b32 v177, v177, v203, v198 bitop3:0xc4\n"
      "v_bitop3_b32 v191, v183, v198, v168 bitop3:0xac\n"
      "v_bitop3_b32 v168, v183, v168, v202 bitop3:0xac\n"
      "v_bitop3_b32 v184, v183, v170, v185 bitop3:0xac\n"
      "v_bitop3_b32 v181, v183, v185, v194 bitop3:0xac\n"
      "v_bitop3_b32 v195, v183, v194, v180 bitop3:0xac\n"
      "v_bitop3_b32 v199, v183, v180, 0 bitop3:0x04\n"
      "v_bitop3_b32 v185, v183, v202, 0 bitop3:0x04\n"
      "v_bitop3_b32 v170, v206, v168, v195 bitop3:0xca\n"
      "v_bitop3_b32 v203, v206, v181, v168 bitop3:0xca\n"
      "v_bitop3_b32 v194, v206, v191, v181 bitop3:0xca\n"
      "v_bitop3_b32 v168, v206, v184, v191 bitop3:0xca\n"
      "v_bitop3_b32 v198, v206, v177, v184 bitop3:0x3a\n"
      "v_bitop3_b32 v202, v206, v177, 0 bitop3:0x04\n"
      "v_bitop3_b32 v177, v206, v195, v185 bitop3:0xca\n"
      "v_bitop3_b32 v180, v206, v185, v199 bitop3:0xca\n"
      "v_bitop3_b32 v210, v206, v199, 0 bitop3:0x40\n"
      "v_bitop3_b32 v181, v171, v202, 0 bitop3:0x10\n"
      "v_bitop3_b32 v169, v202, v169, 0 bitop3:0x04\n"
      "v_bitop3_b32 v180, v177, v180, v210 bitop3:0xfe\n"
      "v_bitop3_b32 v171, v203, v170, 0 bitop3:0x40\n"
      "v_bitop3_b32 v178, v169, v179, v178 bitop3:0xe4\n"
      "v_bitop3_b32 v96, v180, v203, v170 bitop3:0x64\n"
      "v_bitop3_b32 v169, v171, v194, 0 bitop3:0x40\n"
      "v_bitop3_b32 v97, v171, v194, 0 bitop3:0x14\n"
      "v_bitop3_b32 v107, v175, v178, v173 bitop3:0xe4\n"
      "v_bitop3_b32 v171, v169, v168, 0 bitop3:0x40\n"
      "v_bitop3_b32 v101, v169, v168, 0 bitop3:0x14\n"
      "v_bitop3_b32 v175, v183, v174, 0 bitop3:0x14\n"
      "v_bitop3_b32 v170, v183, v174, 0 bitop3:0x54\n"
      "v_bitop3_b32 v169, v171, v198, 0 bitop3:0x40\n"
      "v_bitop3_b32 v99, v171, v198, 0 bitop3:0x14\n"
      "v_bitop3_b32 v168, v169, v206, v176 bitop3:0xe8\n"
      "v_bitop3_b32 v98, v169, v206, v176 bitop3:0x96\n"
      "v_bitop3_b32 v176, v168, v183, v186 bitop3:0xe8\n"
      "v_bitop3_b32 v105, v168, v183, v186 bitop3:0x96\n"
      "v_bitop3_b32 v169, v176, v175, v190 bitop3:0xe8\n"
      "v_bitop3_b32 v102, v176, v175, v190 bitop3:0x96\n"
      "v_bitop3_b32 v168, v169, v170, v172 bitop3:0xe8\n"
      "v_bitop3_b32 v103, v169, v170, v172 bitop3:0x96\n"
      "v_bitop3_b32 v171, v168, v170, v187 bitop3:0xe8\n"
      "v_bitop3_b32 v106, v168, v170, v187 bitop3:0x96\n"
      "v_bitop3_b32 v168, v171, v170, 0 bitop3:0x14\n"
      "v_bitop3_b32 v171, v181, v171, v170 bitop3:0x40\n"
      "v_bitop3_b32 v104, v171, v173, v182 bitop3:0xfe\n"
      "v_bitop3_b32 v100, v181, v182, v168 bitop3:0xdc\n"
      : "+{v96}"(acc[0]), "+{v97}"(acc[1]), "+{v98}"(acc[2]), "+{v99}"(acc[3]), "+{v100}"(acc[4]), "+{v101}"(acc[5]), "+{v102}"(acc[6]), "+{v103}"(acc[7]), "+{v104}"(acc[8]), "+{v105}"(acc[9]), "+{v106}"(acc[10]), "+{v107}"(acc[11])
      : [e] "v"(entry)
      : "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119", "v120", "v121", "v122", "v123", "v124", "v125", "v126", "v127", "v128", "v129", "v130", "v131", "v132", "v133", "v134", "v135", "v136", "v137", "v138", "v139", "v140", "v141", "v142", "v143", "v144", "v145", "v146", "v147", "v148", "v149", "v150", "v151", "v152", "v153", "v154", "v155", "v156", "v157", "v158", "v159", "v160", "v161", "v162", "v163", "v164", "v165", "v166", "v167", "v168", "v169", "v170", "v171", "v172", "v173", "v174", "v175", "v176", "v177", "v178", "v179", "v180", "v181", "v182", "v183", "v184", "v185", "v186", "v187", "v189", "v190", "v191", "v193", "v194", "v195", "v198", "v199", "v202", "v203", "v206", "v207", "v210", "v214", "v218", "v222", "memory");
}
static constexpr int kWSlot[11] = {1, 5, 3, 7, 0, 2, 4, 8, 6, 9, 11};
// K products of one batch (taps c .. c+K-1 of one channel word): the weight rows
// from LDS (row k at wrow + k*12 words), bit c+k of each IFM word, the
// multiplier netlist, 16-byte stores to this lane's ring entries.
static __device__ __forceinline__ void product_batch(const uint32_t (&xw)[11], int c,
                                                     const lds_u32* wrow, lds_u32* entry) {
  asm volatile(
      "ds_read_b128 v[96:99], %[wr] offset:0\n"
      "ds_read_b128 v[100:103], %[wr] offset:16\n"
      "ds_read_b128 v[104:107], %[wr] offset:32\n"
      "ds_read_b128 v[108:111], %[wr] offset:48\n"
      "ds_read_b128 v[112:115], %[wr] offset:64\n"
      "ds_read_b128 v[116:119], %[wr] offset:80\n"
      "ds_read_b128 v[120:123], %[wr] offset:96\n"
      "ds_read_b128 v[124:127], %[wr] offset:112\n"
      "ds_read_b128 v[128:131], %[wr] offset:128\n"
      "ds_read_b128 v[132:135], %[wr] offset:144\n"
      "ds_read_b128 v[136:139], %[wr] offset:160\n"
      "ds_read_b128 v[140:143], %[wr] offset:176\n"
      "v_bfe_i32 v170, %[x0], %[c0], 1\n"
      "v_bfe_i32 v168, %[x1], %[c0], 1\n"
      "v_bfe_i32 v174, %[x2], %[c0], 1\n"
      "v_bfe_i32 v169, %[x3], %[c0], 1\n"
      "v_bfe_i32 v173, %[x4], %[c0], 1\n"
      "v_bfe_i32 v177, %[x5], %[c0], 1\n"
      "v_bfe_i32 v178, %[x6], %[c0], 1\n"
      "v_bfe_i32 v171, %[x7], %[c0], 1\n"
      "v_bfe_i32 v172, %[x8], %[c0], 1\n"
      "v_bfe_i32 v175, %[x9], %[c0], 1\n"
      "v_bfe_i32 v176, %[x10], %[c0], 1\n"
      "s_waitcnt lgkmcnt(9)\n"
      "v_bitop3_b32 v148, v172, v102, 0 bitop3:0x14\n"
      "v_bitop3_b32 v181, v174, v97, 0 bitop3:0x40\n"
      "v_bitop3_b32 v182, v170, v101, 0 bitop3:0x40\n"
      "v_bitop3_b32 v186, v168, v101, 0 bitop3:0x40\n"
      "v_bitop3_b32 v180, v174, v101, 0 bitop3:0x40\n"
      "v_bitop3_b32 v179, v170, v99, 0 bitop3:0x40\n"
      "v_bitop3_b32 v190, v168, v99, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v174, v99, 0 bitop3:0x40\n"
      "v_bitop3_b32 v185, v179, v186, v181 bitop3:0x96\n"
      "v_bitop3_b32 v181, v179, v186, v181 bitop3:0xe8\n"
      "v_bitop3_b32 v179, v190, v180, v97 bitop3:0x96\n"
      "v_bitop3_b32 v180, v190, v180, v97 bitop3:0xe8\n"
      "v_bitop3_b32 v186, v182, v168, v97 bitop3:0x80\n"
      "v_bitop3_b32 v182, v182, v168, v97 bitop3:0x78\n"
      "v_bitop3_b32 v189, v183, v168, v101 bitop3:0x96\n"
      "v_bitop3_b32 v184, v183, v168, v101 bitop3:0xe8\n"
      "v_bitop3_b32 v193, v179, v181, v170 bitop3:0x96\n"
      "v_bitop3_b32 v190, v179, v181, v170 bitop3:0xe8\n"
      "v_bitop3_b32 v179, v186, v185, 0 bitop3:0x40\n"
      "v_bitop3_b32 v188, v186, v185, 0 bitop3:0x14\n"
      "v_bitop3_b32 v192, v190, v189, v180 bitop3:0x96\n"
      "v_bitop3_b32 v180, v190, v189, v180 bitop3:0xe8\n"
      "v_bitop3_b32 v181, v179, v193, 0 bitop3:0x40\n"
      "v_bitop3_b32 v179, v179, v193, 0 bitop3:0x14\n"
      "v_bitop3_b32 v183, v184, v174, v99 bitop3:0x96\n"
      "v_bitop3_b32 v185, v184, v174, v99 bitop3:0xe8\n"
      "v_bitop3_b32 v189, v181, v192, 0 bitop3:0x40\n"
      "v_bitop3_b32 v186, v181, v192, 0 bitop3:0x14\n"
      "v_bitop3_b32 v184, v176, v175, 0 bitop3:0x40\n"
      "v_bitop3_b32 v187, v189, v180, v183 bitop3:0xe8\n"
      "v_bitop3_b32 v180, v189, v180, v183 bitop3:0x96\n"
      "v_bitop3_b32 v181, v184, v107, v105 bitop3:0xf8\n"
      "v_bitop3_b32 v189, v187, v185, 0 bitop3:0x54\n"
      "v_bitop3_b32 v184, v187, v180, v185 bitop3:0xa4\n"
      "v_bitop3_b32 v190, v176, v175, 0 bitop3:0x10\n"
      "v_bitop3_b32 v180, v189, v180, v186 bitop3:0xca\n"
      "v_bitop3_b32 v186, v189, v186, v179 bitop3:0xca\n"
      "v_bitop3_b32 v194, v189, v179, v188 bitop3:0xca\n"
      "v_bitop3_b32 v179, v189, v188, v182 bitop3:0xca\n"
      "v_bitop3_b32 v183, v189, v182, 0 bitop3:0x40\n"
      "v_bitop3_b32 v188, v176, v175, 0 bitop3:0x54\n"
      "v_bitop3_b32 v182, v176, v175, 0 bitop3:0x04\n"
      "v_bitop3_b32 v192, v183, v170, v97 bitop3:0xf8\n"
      "v_bitop3_b32 v198, v188, v107, v105 bitop3:0x04\n"
      "v_bitop3_b32 v185, v182, v107, v105 bitop3:0x20\n"
      "v_bitop3_b32 v144, v192, v179, v194 bitop3:0x62\n"
      "v_bitop3_b32 v179, v179, v194, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v190, v107, v105 bitop3:0x10\n"
      "v_bitop3_b32 v193, v190, v107, v105 bitop3:0xf4\n"
      "v_bitop3_b32 v197, v179, v186, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v183, v198, v181 bitop3:0xfe\n"
      "v_bitop3_b32 v146, v179, v186, 0 bitop3:0x14\n"
      "v_bitop3_b32 v182, v197, v180, 0 bitop3:0x40\n"
      "v_bitop3_b32 v150, v197, v180, 0 bitop3:0x14\n"
      "v_bitop3_b32 v186, v182, v184, v189 bitop3:0xea\n"
      "v_bitop3_b32 v145, v182, v184, 0 bitop3:0x14\n"
      "v_bitop3_b32 v179, v186, v169, v103 bitop3:0xe8\n"
      "v_bitop3_b32 v147, v186, v169, v103 bitop3:0x69\n"
      "v_bitop3_b32 v180, v179, v173, v96 bitop3:0x96\n"
      "v_bitop3_b32 v179, v179, v173, v96 bitop3:0xe8\n"
      "v_bitop3_b32 v182, v179, v177, v98 bitop3:0x96\n"
      "v_bitop3_b32 v187, v180, v147, 0 bitop3:0x10\n"
      "v_bitop3_b32 v181, v179, v177, v98 bitop3:0xe8\n"
      "v_bitop3_b32 v154, v180, v147, 0 bitop3:0x41\n"
      "v_bitop3_b32 v189, v187, v182, 0 bitop3:0x40\n"
      "v_bitop3_b32 v149, v187, v182, 0 bitop3:0x14\n"
      "v_bitop3_b32 v180, v181, v178, v100 bitop3:0x96\n"
      "v_bitop3_b32 v181, v181, v178, v100 bitop3:0xe8\n"
      "v_bitop3_b32 v182, v181, v171, v104 bitop3:0x96\n"
      "v_bitop3_b32 v179, v189, v180, 0 bitop3:0x40\n"
      "v_bitop3_b32 v187, v181, v171, v104 bitop3:0xe8\n"
      "v_bitop3_b32 v153, v189, v180, 0 bitop3:0x14\n"
      "v_bitop3_b32 v186, v179, v182, 0 bitop3:0x54\n"
      "v_bitop3_b32 v151, v179, v182, 0 bitop3:0x41\n"
      "v_bitop3_b32 v180, v186, v187, 0 bitop3:0x14\n"
      "v_bitop3_b32 v184, v185, v186, v187 bitop3:0x80\n"
      "v_bitop3_b32 v152, v184, v193, v183 bitop3:0xfe\n"
      "v_bitop3_b32 v155, v183, v185, v180 bitop3:0xf8\n"
      "s_nop 4\n"
      "ds_write_b128 %[e], v[144:147] offset:0\n"
      "ds_write_b128 %[e], v[148:151] offset:16\n"
      "ds_write_b128 %[e], v[152:155] offset:32\n"
      "v_bfe_i32 v170, %[x0], %[c1], 1\n"
      "v_bfe_i32 v168, %[x1], %[c1], 1\n"
      "v_bfe_i32 v174, %[x2], %[c1], 1\n"
      "v_bfe_i32 v169, %[x3], %[c1], 1\n"
      "v_bfe_i32 v173, %[x4], %[c1], 1\n"
      "v_bfe_i32 v177, %[x5], %[c1], 1\n"
      "v_bfe_i32 v178, %[x6], %[c1], 1\n"
      "v_bfe_i32 v171, %[x7], %[c1], 1\n"
      "v_bfe_i32 v172, %[x8], %[c1], 1\n"
      "v_bfe_i32 v175, %[x9], %[c1], 1\n"
      "v_bfe_i32 v176, %[x10], %[c1], 1\n"
      "s_waitcnt lgkmcnt(9)\n"
      "v_bitop3_b32 v160, v172, v114, 0 bitop3:0x14\n"
      "v_bitop3_b32 v181, v174, v109, 0 bitop3:0x40\n"
      "v_bitop3_b32 v182, v170, v113, 0 bitop3:0x40\n"
      "v_bitop3_b32 v186, v168, v113, 0 bitop3:0x40\n"
      "v_bitop3_b32 v180, v174, v113, 0 bitop3:0x40\n"
      "v_bitop3_b32 v179, v170, v111, 0 bitop3:0x40\n"
      "v_bitop3_b32 v190, v168, v111, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v174, v111, 0 bitop3:0x40\n"
      "v_bitop3_b32 v185, v179, v186, v181 bitop3:0x96\n"
      "v_bitop3_b32 v181, v179, v186, v181 bitop3:0xe8\n"
      "v_bitop3_b32 v179, v190, v180, v109 bitop3:0x96\n"
      "v_bitop3_b32 v180, v190, v180, v109 bitop3:0xe8\n"
      "v_bitop3_b32 v186, v182, v168, v109 bitop3:0x80\n"
      "v_bitop3_b32 v182, v182, v168, v109 bitop3:0x78\n"
      "v_bitop3_b32 v189, v183, v168, v113 bitop3:0x96\n"
      "v_bitop3_b32 v184, v183, v168, v113 bitop3:0xe8\n"
      "v_bitop3_b32 v193, v179, v181, v170 bitop3:0x96\n"
      "v_bitop3_b32 v190, v179, v181, v170 bitop3:0xe8\n"
      "v_bitop3_b32 v179, v186, v185, 0 bitop3:0x40\n"
      "v_bitop3_b32 v188, v186, v185, 0 bitop3:0x14\n"
      "v_bitop3_b32 v192, v190, v189, v180 bitop3:0x96\n"
      "v_bitop3_b32 v180, v190, v189, v180 bitop3:0xe8\n"
      "v_bitop3_b32 v181, v179, v193, 0 bitop3:0x40\n"
      "v_bitop3_b32 v179, v179, v193, 0 bitop3:0x14\n"
      "v_bitop3_b32 v183, v184, v174, v111 bitop3:0x96\n"
      "v_bitop3_b32 v185, v184, v174, v111 bitop3:0xe8\n"
      "v_bitop3_b32 v189, v181, v192, 0 bitop3:0x40\n"
      "v_bitop3_b32 v186, v181, v192, 0 bitop3:0x14\n"
      "v_bitop3_b32 v184, v176, v175, 0 bitop3:0x40\n"
      "v_bitop3_b32 v187, v189, v180, v183 bitop3:0xe8\n"
      "v_bitop3_b32 v180, v189, v180, v183 bitop3:0x96\n"
      "v_bitop3_b32 v181, v184, v119, v117 bitop3:0xf8\n"
      "v_bitop3_b32 v189, v187, v185, 0 bitop3:0x54\n"
      "v_bitop3_b32 v184, v187, v180, v185 bitop3:0xa4\n"
      "v_bitop3_b32 v190, v176, v175, 0 bitop3:0x10\n"
      "v_bitop3_b32 v180, v189, v180, v186 bitop3:0xca\n"
      "v_bitop3_b32 v186, v189, v186, v179 bitop3:0xca\n"
      "v_bitop3_b32 v194, v189, v179, v188 bitop3:0xca\n"
      "v_bitop3_b32 v179, v189, v188, v182 bitop3:0xca\n"
      "v_bitop3_b32 v183, v189, v182, 0 bitop3:0x40\n"
      "v_bitop3_b32 v188, v176, v175, 0 bitop3:0x54\n"
      "v_bitop3_b32 v182, v176, v175, 0 bitop3:0x04\n"
      "v_bitop3_b32 v192, v183, v170, v109 bitop3:0xf8\n"
      "v_bitop3_b32 v198, v188, v119, v117 bitop3:0x04\n"
      "v_bitop3_b32 v185, v182, v119, v117 bitop3:0x20\n"
      "v_bitop3_b32 v156, v192, v179, v194 bitop3:0x62\n"
      "v_bitop3_b32 v179, v179, v194, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v190, v119, v117 bitop3:0x10\n"
      "v_bitop3_b32 v193, v190, v119, v117 bitop3:0xf4\n"
      "v_bitop3_b32 v197, v179, v186, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v183, v198, v181 bitop3:0xfe\n"
      "v_bitop3_b32 v158, v179, v186, 0 bitop3:0x14\n"
      "v_bitop3_b32 v182, v197, v180, 0 bitop3:0x40\n"
      "v_bitop3_b32 v162, v197, v180, 0 bitop3:0x14\n"
      "v_bitop3_b32 v186, v182, v184, v189 bitop3:0xea\n"
      "v_bitop3_b32 v157, v182, v184, 0 bitop3:0x14\n"
      "v_bitop3_b32 v179, v186, v169, v115 bitop3:0xe8\n"
      "v_bitop3_b32 v159, v186, v169, v115 bitop3:0x69\n"
      "v_bitop3_b32 v180, v179, v173, v108 bitop3:0x96\n"
      "v_bitop3_b32 v179, v179, v173, v108 bitop3:0xe8\n"
      "v_bitop3_b32 v182, v179, v177, v110 bitop3:0x96\n"
      "v_bitop3_b32 v187, v180, v159, 0 bitop3:0x10\n"
      "v_bitop3_b32 v181, v179, v177, v110 bitop3:0xe8\n"
      "v_bitop3_b32 v166, v180, v159, 0 bitop3:0x41\n"
      "v_bitop3_b32 v189, v187, v182, 0 bitop3:0x40\n"
      "v_bitop3_b32 v161, v187, v182, 0 bitop3:0x14\n"
      "v_bitop3_b32 v180, v181, v178, v112 bitop3:0x96\n"
      "v_bitop3_b32 v181, v181, v178, v112 bitop3:0xe8\n"
      "v_bitop3_b32 v182, v181, v171, v116 bitop3:0x96\n"
      "v_bitop3_b32 v179, v189, v180, 0 bitop3:0x40\n"
      "v_bitop3_b32 v187, v181, v171, v116 bitop3:0xe8\n"
      "v_bitop3_b32 v165, v189, v180, 0 bitop3:0x14\n"
      "v_bitop3_b32 v186, v179, v182, 0 bitop3:0x54\n"
      "v_bitop3_b32 v163, v179, v182, 0 bitop3:0x41\n"
      "v_bitop3_b32 v180, v186, v187, 0 bitop3:0x14\n"
      "v_bitop3_b32 v184, v185, v186, v187 bitop3:0x80\n"
      "v_bitop3_b32 v164, v184, v193, v183 bitop3:0xfe\n"
      "v_bitop3_b32 v167, v183, v185, v180 bitop3:0xf8\n"
      "s_nop 4\n"
      "ds_write_b128 %[e], v[156:159] offset:12288\n"
      "ds_write_b128 %[e], v[160:163] offset:12304\n"
      "ds_write_b128 %[e], v[164:167] offset:12320\n"
      "v_bfe_i32 v170, %[x0], %[c2], 1\n"
      "v_bfe_i32 v168, %[x1], %[c2], 1\n"
      "v_bfe_i32 v174, %[x2], %[c2], 1\n"
      "v_bfe_i32 v169, %[x3], %[c2], 1\n"
      "v_bfe_i32 v173, %[x4], %[c2], 1\n"
      "v_bfe_i32 v177, %[x5], %[c2], 1\n"
      "v_bfe_i32 v178, %[x6], %[c2], 1\n"
      "v_bfe_i32 v171, %[x7], %[c2], 1\n"
      "v_bfe_i32 v172, %[x8], %[c2], 1\n"
      "v_bfe_i32 v175, %[x9], %[c2], 1\n"
      "v_bfe_i32 v176, %[x10], %[c2], 1\n"
      "s_waitcnt lgkmcnt(3)\n"
      "v_bitop3_b32 v148, v172, v126, 0 bitop3:0x14\n"
      "v_bitop3_b32 v181, v174, v121, 0 bitop3:0x40\n"
      "v_bitop3_b32 v182, v170, v125, 0 bitop3:0x40\n"
      "v_bitop3_b32 v186, v168, v125, 0 bitop3:0x40\n"
      "v_bitop3_b32 v180, v174, v125, 0 bitop3:0x40\n"
      "v_bitop3_b32 v179, v170, v123, 0 bitop3:0x40\n"
      "v_bitop3_b32 v190, v168, v123, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v174, v123, 0 bitop3:0x40\n"
      "v_bitop3_b32 v185, v179, v186, v181 bitop3:0x96\n"
      "v_bitop3_b32 v181, v179, v186, v181 bitop3:0xe8\n"
      "v_bitop3_b32 v179, v190, v180, v121 bitop3:0x96\n"
      "v_bitop3_b32 v180, v190, v180, v121 bitop3:0xe8\n"
      "v_bitop3_b32 v186, v182, v168, v121 bitop3:0x80\n"
      "v_bitop3_b32 v182, v182, v168, v121 bitop3:0x78\n"
      "v_bitop3_b32 v189, v183, v168, v125 bitop3:0x96\n"
      "v_bitop3_b32 v184, v183, v168, v125 bitop3:0xe8\n"
      "v_bitop3_b32 v193, v179, v181, v170 bitop3:0x96\n"
      "v_bitop3_b32 v190, v179, v181, v170 bitop3:0xe8\n"
      "v_bitop3_b32 v179, v186, v185, 0 bitop3:0x40\n"
      "v_bitop3_b32 v188, v186, v185, 0 bitop3:0x14\n"
      "v_bitop3_b32 v192, v190, v189, v180 bitop3:0x96\n"
      "v_bitop3_b32 v180, v190, v189, v180 bitop3:0xe8\n"
      "v_bitop3_b32 v181, v179, v193, 0 bitop3:0x40\n"
      "v_bitop3_b32 v179, v179, v193, 0 bitop3:0x14\n"
      "v_bitop3_b32 v183, v184, v174, v123 bitop3:0x96\n"
      "v_bitop3_b32 v185, v184, v174, v123 bitop3:0xe8\n"
      "v_bitop3_b32 v189, v181, v192, 0 bitop3:0x40\n"
      "v_bitop3_b32 v186, v181, v192, 0 bitop3:0x14\n"
      "v_bitop3_b32 v184, v176, v175, 0 bitop3:0x40\n"
      "v_bitop3_b32 v187, v189, v180, v183 bitop3:0xe8\n"
      "v_bitop3_b32 v180, v189, v180, v183 bitop3:0x96\n"
      "v_bitop3_b32 v181, v184, v131, v129 bitop3:0xf8\n"
      "v_bitop3_b32 v189, v187, v185, 0 bitop3:0x54\n"
      "v_bitop3_b32 v184, v187, v180, v185 bitop3:0xa4\n"
      "v_bitop3_b32 v190, v176, v175, 0 bitop3:0x10\n"
      "v_bitop3_b32 v180, v189, v180, v186 bitop3:0xca\n"
      "v_bitop3_b32 v186, v189, v186, v179 bitop3:0xca\n"
      "v_bitop3_b32 v194, v189, v179, v188 bitop3:0xca\n"
      "v_bitop3_b32 v179, v189, v188, v182 bitop3:0xca\n"
      "v_bitop3_b32 v183, v189, v182, 0 bitop3:0x40\n"
      "v_bitop3_b32 v188, v176, v175, 0 bitop3:0x54\n"
      "v_bitop3_b32 v182, v176, v175, 0 bitop3:0x04\n"
      "v_bitop3_b32 v192, v183, v170, v121 bitop3:0xf8\n"
      "v_bitop3_b32 v198, v188, v131, v129 bitop3:0x04\n"
      "v_bitop3_b32 v185, v182, v131, v129 bitop3:0x20\n"
      "v_bitop3_b32 v144, v192, v179, v194 bitop3:0x62\n"
      "v_bitop3_b32 v179, v179, v194, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v190, v131, v129 bitop3:0x10\n"
      "v_bitop3_b32 v193, v190, v131, v129 bitop3:0xf4\n"
      "v_bitop3_b32 v197, v179, v186, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v183, v198, v181 bitop3:0xfe\n"
      "v_bitop3_b32 v146, v179, v186, 0 bitop3:0x14\n"
      "v_bitop3_b32 v182, v197, v180, 0 bitop3:0x40\n"
      "v_bitop3_b32 v150, v197, v180, 0 bitop3:0x14\n"
      "v_bitop3_b32 v186, v182, v184, v189 bitop3:0xea\n"
      "v_bitop3_b32 v145, v182, v184, 0 bitop3:0x14\n"
      "v_bitop3_b32 v179, v186, v169, v127 bitop3:0xe8\n"
      "v_bitop3_b32 v147, v186, v169, v127 bitop3:0x69\n"
      "v_bitop3_b32 v180, v179, v173, v120 bitop3:0x96\n"
      "v_bitop3_b32 v179, v179, v173, v120 bitop3:0xe8\n"
      "v_bitop3_b32 v182, v179, v177, v122 bitop3:0x96\n"
      "v_bitop3_b32 v187, v180, v147, 0 bitop3:0x10\n"
      "v_bitop3_b32 v181, v179, v177, v122 bitop3:0xe8\n"
      "v_bitop3_b32 v154, v180, v147, 0 bitop3:0x41\n"
      "v_bitop3_b32 v189, v187, v182, 0 bitop3:0x40\n"
      "v_bitop3_b32 v149, v187, v182, 0 bitop3:0x14\n"
      "v_bitop3_b32 v180, v181, v178, v124 bitop3:0x96\n"
      "v_bitop3_b32 v181, v181, v178, v124 bitop3:0xe8\n"
      "v_bitop3_b32 v182, v181, v171, v128 bitop3:0x96\n"
      "v_bitop3_b32 v179, v189, v180, 0 bitop3:0x40\n"
      "v_bitop3_b32 v187, v181, v171, v128 bitop3:0xe8\n"
      "v_bitop3_b32 v153, v189, v180, 0 bitop3:0x14\n"
      "v_bitop3_b32 v186, v179, v182, 0 bitop3:0x54\n"
      "v_bitop3_b32 v151, v179, v182, 0 bitop3:0x41\n"
      "v_bitop3_b32 v180, v186, v187, 0 bitop3:0x14\n"
      "v_bitop3_b32 v184, v185, v186, v187 bitop3:0x80\n"
      "v_bitop3_b32 v152, v184, v193, v183 bitop3:0xfe\n"
      "v_bitop3_b32 v155, v183, v185, v180 bitop3:0xf8\n"
      "s_nop 4\n"
      "ds_write_b128 %[e], v[144:147] offset:24576\n"
      "ds_write_b128 %[e], v[148:151] offset:24592\n"
      "ds_write_b128 %[e], v[152:155] offset:24608\n"
      "v_bfe_i32 v170, %[x0], %[c3], 1\n"
      "v_bfe_i32 v168, %[x1], %[c3], 1\n"
      "v_bfe_i32 v174, %[x2], %[c3], 1\n"
      "v_bfe_i32 v169, %[x3], %[c3], 1\n"
      "v_bfe_i32 v173, %[x4], %[c3], 1\n"
      "v_bfe_i32 v177, %[x5], %[c3], 1\n"
      "v_bfe_i32 v178, %[x6], %[c3], 1\n"
      "v_bfe_i32 v171, %[x7], %[c3], 1\n"
      "v_bfe_i32 v172, %[x8], %[c3], 1\n"
      "v_bfe_i32 v175, %[x9], %[c3], 1\n"
      "v_bfe_i32 v176, %[x10], %[c3], 1\n"
      "s_waitcnt lgkmcnt(3)\n"
      "v_bitop3_b32 v160, v172, v138, 0 bitop3:0x14\n"
      "v_bitop3_b32 v181, v174, v133, 0 bitop3:0x40\n"
      "v_bitop3_b32 v182, v170, v137, 0 bitop3:0x40\n"
      "v_bitop3_b32 v186, v168, v137, 0 bitop3:0x40\n"
      "v_bitop3_b32 v180, v174, v137, 0 bitop3:0x40\n"
      "v_bitop3_b32 v179, v170, v135, 0 bitop3:0x40\n"
      "v_bitop3_b32 v190, v168, v135, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v174, v135, 0 bitop3:0x40\n"
      "v_bitop3_b32 v185, v179, v186, v181 bitop3:0x96\n"
      "v_bitop3_b32 v181, v179, v186, v181 bitop3:0xe8\n"
      "v_bitop3_b32 v179, v190, v180, v133 bitop3:0x96\n"
      "v_bitop3_b32 v180, v190, v180, v133 bitop3:0xe8\n"
      "v_bitop3_b32 v186, v182, v168, v133 bitop3:0x80\n"
      "v_bitop3_b32 v182, v182, v168, v133 bitop3:0x78\n"
      "v_bitop3_b32 v189, v183, v168, v137 bitop3:0x96\n"
      "v_bitop3_b32 v184, v183, v168, v137 bitop3:0xe8\n"
      "v_bitop3_b32 v193, v179, v181, v170 bitop3:0x96\n"
      "v_bitop3_b32 v190, v179, v181, v170 bitop3:0xe8\n"
      "v_bitop3_b32 v179, v186, v185, 0 bitop3:0x40\n"
      "v_bitop3_b32 v188, v186, v185, 0 bitop3:0x14\n"
      "v_bitop3_b32 v192, v190, v189, v180 bitop3:0x96\n"
      "v_bitop3_b32 v180, v190, v189, v180 bitop3:0xe8\n"
      "v_bitop3_b32 v181, v179, v193, 0 bitop3:0x40\n"
      "v_bitop3_b32 v179, v179, v193, 0 bitop3:0x14\n"
      "v_bitop3_b32 v183, v184, v174, v135 bitop3:0x96\n"
      "v_bitop3_b32 v185, v184, v174, v135 bitop3:0xe8\n"
      "v_bitop3_b32 v189, v181, v192, 0 bitop3:0x40\n"
      "v_bitop3_b32 v186, v181, v192, 0 bitop3:0x14\n"
      "v_bitop3_b32 v184, v176, v175, 0 bitop3:0x40\n"
      "v_bitop3_b32 v187, v189, v180, v183 bitop3:0xe8\n"
      "v_bitop3_b32 v180, v189, v180, v183 bitop3:0x96\n"
      "v_bitop3_b32 v181, v184, v143, v141 bitop3:0xf8\n"
      "v_bitop3_b32 v189, v187, v185, 0 bitop3:0x54\n"
      "v_bitop3_b32 v184, v187, v180, v185 bitop3:0xa4\n"
      "v_bitop3_b32 v190, v176, v175, 0 bitop3:0x10\n"
      "v_bitop3_b32 v180, v189, v180, v186 bitop3:0xca\n"
      "v_bitop3_b32 v186, v189, v186, v179 bitop3:0xca\n"
      "v_bitop3_b32 v194, v189, v179, v188 bitop3:0xca\n"
      "v_bitop3_b32 v179, v189, v188, v182 bitop3:0xca\n"
      "v_bitop3_b32 v183, v189, v182, 0 bitop3:0x40\n"
      "v_bitop3_b32 v188, v176, v175, 0 bitop3:0x54\n"
      "v_bitop3_b32 v182, v176, v175, 0 bitop3:0x04\n"
      "v_bitop3_b32 v192, v183, v170, v133 bitop3:0xf8\n"
      "v_bitop3_b32 v198, v188, v143, v141 bitop3:0x04\n"
      "v_bitop3_b32 v185, v182, v143, v141 bitop3:0x20\n"
      "v_bitop3_b32 v156, v192, v179, v194 bitop3:0x62\n"
      "v_bitop3_b32 v179, v179, v194, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v190, v143, v141 bitop3:0x10\n"
      "v_bitop3_b32 v193, v190, v143, v141 bitop3:0xf4\n"
      "v_bitop3_b32 v197, v179, v186, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v183, v198, v181 bitop3:0xfe\n"
      "v_bitop3_b32 v158, v179, v186, 0 bitop3:0x14\n"
      "v_bitop3_b32 v182, v197, v180, 0 bitop3:0x40\n"
      "v_bitop3_b32 v162, v197, v180, 0 bitop3:0x14\n"
      "v_bitop3_b32 v186, v182, v184, v189 bitop3:0xea\n"
      "v_bitop3_b32 v157, v182, v184, 0 bitop3:0x14\n"
      "v_bitop3_b32 v179, v186, v169, v139 bitop3:0xe8\n"
      "v_bitop3_b32 v159, v186, v169, v139 bitop3:0x69\n"
      "v_bitop3_b32 v180, v179, v173, v132 bitop3:0x96\n"
      "v_bitop3_b32 v179, v179, v173, v132 bitop3:0xe8\n"
      "v_bitop3_b32 v182, v179, v177, v134 bitop3:0x96\n"
      "v_bitop3_b32 v187, v180, v159, 0 bitop3:0x10\n"
      "v_bitop3_b32 v181, v179, v177, v134 bitop3:0xe8\n"
      "v_bitop3_b32 v166, v180, v159, 0 bitop3:0x41\n"
      "v_bitop3_b32 v189, v187, v182, 0 bitop3:0x40\n"
      "v_bitop3_b32 v161, v187, v182, 0 bitop3:0x14\n"
      "v_bitop3_b32 v180, v181, v178, v136 bitop3:0x96\n"
      "v_bitop3_b32 v181, v181, v178, v136 bitop3:0xe8\n"
      "v_bitop3_b32 v182, v181, v171, v140 bitop3:0x96\n"
      "v_bitop3_b32 v179, v189, v180, 0 bitop3:0x40\n"
      "v_bitop3_b32 v187, v181, v171, v140 bitop3:0xe8\n"
      "v_bitop3_b32 v165, v189, v180, 0 bitop3:0x14\n"
      "v_bitop3_b32 v186, v179, v182, 0 bitop3:0x54\n"
      "v_bitop3_b32 v163, v179, v182, 0 bitop3:0x41\n"
      "v_bitop3_b32 v180, v186, v187, 0 bitop3:0x14\n"
      "v_bitop3_b32 v184, v185, v186, v187 bitop3:0x80\n"
      "v_bitop3_b32 v164, v184, v193, v183 bitop3:0xfe\n"
      "v_bitop3_b32 v167, v183, v185, v180 bitop3:0xf8\n"
      "s_nop 4\n"
      "ds_write_b128 %[e], v[156:159] offset:36864\n"
      "ds_write_b128 %[e], v[160:163] offset:36880\n"
      "ds_write_b128 %[e], v[164:167] offset:36896\n"
      :
      : [x0] "v"(xw[0]), [x1] "v"(xw[1]), [x2] "v"(xw[2]), [x3] "v"(xw[3]), [x4] "v"(xw[4]), [x5] "v"(xw[5]), [x6] "v"(xw[6]), [x7] "v"(xw[7]), [x8] "v"(xw[8]), [x9] "v"(xw[9]), [x10] "v"(xw[10]), [c0] "s"(c + 0), [c1] "s"(c + 1), [c2] "s"(c + 2), [c3] "s"(c + 3), [wr] "v"(wrow), [e] "v"(entry)
      : "v96", "v97", "v98", "v99", "v100", "v101", "v102", "v103", "v104", "v105", "v106", "v107", "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119", "v120", "v121", "v122", "v123", "v124", "v125", "v126", "v127", "v128", "v129", "v130", "v131", "v132", "v133", "v134", "v135", "v136", "v137", "v138", "v139", "v140", "v141", "v142", "v143", "v144", "v145", "v146", "v147", "v148", "v149", "v150", "v151", "v152", "v153", "v154", "v155", "v156", "v157", "v158", "v159", "v160", "v161", "v162", "v163", "v164", "v165", "v166", "v167", "v168", "v169", "v170", "v171", "v172", "v173", "v174", "v175", "v176", "v177", "v178", "v179", "v180", "v181", "v182", "v183", "v184", "v185", "v186", "v187", "v188", "v189", "v190", "v192", "v193", "v194", "v197", "v198", "memory");
}
// One product (tap c).
static __device__ __forceinline__ void product_step(const uint32_t (&xw)[11], int c,
                                                    const lds_u32* wrow, lds_u32* entry) {
  asm volatile(
      "ds_read_b128 v[96:99], %[wr] offset:0\n"
      "ds_read_b128 v[100:103], %[wr] offset:16\n"
      "ds_read_b128 v[104:107], %[wr] offset:32\n"
      "v_bfe_i32 v170, %[x0], %[c0], 1\n"
      "v_bfe_i32 v168, %[x1], %[c0], 1\n"
      "v_bfe_i32 v174, %[x2], %[c0], 1\n"
      "v_bfe_i32 v169, %[x3], %[c0], 1\n"
      "v_bfe_i32 v173, %[x4], %[c0], 1\n"
      "v_bfe_i32 v177, %[x5], %[c0], 1\n"
      "v_bfe_i32 v178, %[x6], %[c0], 1\n"
      "v_bfe_i32 v171, %[x7], %[c0], 1\n"
      "v_bfe_i32 v172, %[x8], %[c0], 1\n"
      "v_bfe_i32 v175, %[x9], %[c0], 1\n"
      "v_bfe_i32 v176, %[x10], %[c0], 1\n"
      "s_waitcnt lgkmcnt(0)\n"
      "v_bitop3_b32 v148, v172, v102, 0 bitop3:0x14\n"
      "v_bitop3_b32 v181, v174, v97, 0 bitop3:0x40\n"
      "v_bitop3_b32 v182, v170, v101, 0 bitop3:0x40\n"
      "v_bitop3_b32 v186, v168, v101, 0 bitop3:0x40\n"
      "v_bitop3_b32 v180, v174, v101, 0 bitop3:0x40\n"
      "v_bitop3_b32 v179, v170, v99, 0 bitop3:0x40\n"
      "v_bitop3_b32 v190, v168, v99, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v174, v99, 0 bitop3:0x40\n"
      "v_bitop3_b32 v185, v179, v186, v181 bitop3:0x96\n"
      "v_bitop3_b32 v181, v179, v186, v181 bitop3:0xe8\n"
      "v_bitop3_b32 v179, v190, v180, v97 bitop3:0x96\n"
      "v_bitop3_b32 v180, v190, v180, v97 bitop3:0xe8\n"
      "v_bitop3_b32 v186, v182, v168, v97 bitop3:0x80\n"
      "v_bitop3_b32 v182, v182, v168, v97 bitop3:0x78\n"
      "v_bitop3_b32 v189, v183, v168, v101 bitop3:0x96\n"
      "v_bitop3_b32 v184, v183, v168, v101 bitop3:0xe8\n"
      "v_bitop3_b32 v193, v179, v181, v170 bitop3:0x96\n"
      "v_bitop3_b32 v190, v179, v181, v170 bitop3:0xe8\n"
      "v_bitop3_b32 v179, v186, v185, 0 bitop3:0x40\n"
      "v_bitop3_b32 v188, v186, v185, 0 bitop3:0x14\n"
      "v_bitop3_b32 v192, v190, v189, v180 bitop3:0x96\n"
      "v_bitop3_b32 v180, v190, v189, v180 bitop3:0xe8\n"
      "v_bitop3_b32 v181, v179, v193, 0 bitop3:0x40\n"
      "v_bitop3_b32 v179, v179, v193, 0 bitop3:0x14\n"
      "v_bitop3_b32 v183, v184, v174, v99 bitop3:0x96\n"
      "v_bitop3_b32 v185, v184, v174, v99 bitop3:0xe8\n"
      "v_bitop3_b32 v189, v181, v192, 0 bitop3:0x40\n"
      "v_bitop3_b32 v186, v181, v192, 0 bitop3:0x14\n"
      "v_bitop3_b32 v184, v176, v175, 0 bitop3:0x40\n"
      "v_bitop3_b32 v187, v189, v180, v183 bitop3:0xe8\n"
      "v_bitop3_b32 v180, v189, v180, v183 bitop3:0x96\n"
      "v_bitop3_b32 v181, v184, v107, v105 bitop3:0xf8\n"
      "v_bitop3_b32 v189, v187, v185, 0 bitop3:0x54\n"
      "v_bitop3_b32 v184, v187, v180, v185 bitop3:0xa4\n"
      "v_bitop3_b32 v190, v176, v175, 0 bitop3:0x10\n"
      "v_bitop3_b32 v180, v189, v180, v186 bitop3:0xca\n"
      "v_bitop3_b32 v186, v189, v186, v179 bitop3:0xca\n"
      "v_bitop3_b32 v194, v189, v179, v188 bitop3:0xca\n"
      "v_bitop3_b32 v179, v189, v188, v182 bitop3:0xca\n"
      "v_bitop3_b32 v183, v189, v182, 0 bitop3:0x40\n"
      "v_bitop3_b32 v188, v176, v175, 0 bitop3:0x54\n"
      "v_bitop3_b32 v182, v176, v175, 0 bitop3:0x04\n"
      "v_bitop3_b32 v192, v183, v170, v97 bitop3:0xf8\n"
      "v_bitop3_b32 v198, v188, v107, v105 bitop3:0x04\n"
      "v_bitop3_b32 v185, v182, v107, v105 bitop3:0x20\n"
      "v_bitop3_b32 v144, v192, v179, v194 bitop3:0x62\n"
      "v_bitop3_b32 v179, v179, v194, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v190, v107, v105 bitop3:0x10\n"
      "v_bitop3_b32 v193, v190, v107, v105 bitop3:0xf4\n"
      "v_bitop3_b32 v197, v179, v186, 0 bitop3:0x40\n"
      "v_bitop3_b32 v183, v183, v198, v181 bitop3:0xfe\n"
      "v_bitop3_b32 v146, v179, v186, 0 bitop3:0x14\n"
      "v_bitop3_b32 v182, v197, v180, 0 bitop3:0x40\n"
      "v_bitop3_b32 v150, v197, v180, 0 bitop3:0x14\n"
      "v_bitop3_b32 v186, v182, v184, v189 bitop3:0xea\n"
      "v_bitop3_b32 v145, v182, v184, 0 bitop3:0x14\n"
      "v_bitop3_b32 v179, v186, v169, v103 bitop3:0xe8\n"
      "v_bitop3_b32 v147, v186, v169, v103 bitop3:0x69\n"
      "v_bitop3_b32 v180, v179, v173, v96 bitop3:0x96\n"
      "v_bitop3_b32 v179, v179, v173, v96 bitop3:0xe8\n"
      "v_bitop3_b32 v182, v179, v177, v98 bitop3:0x96\n"
      "v_bitop3_b32 v187, v180, v147, 0 bitop3:0x10\n"
      "v_bitop3_b32 v181, v179, v177, v98 bitop3:0xe8\n"
      "v_bitop3_b32 v154, v180, v147, 0 bitop3:0x41\n"
      "v_bitop3_b32 v189, v187, v182, 0 bitop3:0x40\n"
      "v_bitop3_b32 v149, v187, v182, 0 bitop3:0x14\n"
      "v_bitop3_b32 v180, v181, v178, v100 bitop3:0x96\n"
      "v_bitop3_b32 v181, v181, v178, v100 bitop3:0xe8\n"
      "v_bitop3_b32 v182, v181, v171, v104 bitop3:0x96\n"
      "v_bitop3_b32 v179, v189, v180, 0 bitop3:0x40\n"
      "v_bitop3_b32 v187, v181, v171, v104 bitop3:0xe8\n"
      "v_bitop3_b32 v153, v189, v180, 0 bitop3:0x14\n"
      "v_bitop3_b32 v186, v179, v182, 0 bitop3:0x54\n"
      "v_bitop3_b32 v151, v179, v182, 0 bitop3:0x41\n"
      "v_bitop3_b32 v180, v186, v187, 0 bitop3:0x14\n"
      "v_bitop3_b32 v184, v185, v186, v187 bitop3:0x80\n"
      "v_bitop3_b32 v152, v184, v193, v183 bitop3:0xfe\n"
      "v_bitop3_b32 v155, v183, v185, v180 bitop3:0xf8\n"
      "s_nop 4\n"
      "ds_write_b128 %[e], v[144:147] offset:0\n"
      "ds_write_b128 %[e], v[148:151] offset:16\n"
      "ds_write_b128 %[e], v[152:155] offset:32\n"
      :
      : [x0] "v"(xw[0]), [x1] "v"(xw[1]), [x2] "v"(xw[2]), [x3] "v"(xw[3]), [x4] "v"(xw[4]), [x5] "v"(xw[5]), [x6] "v"(xw[6]), [x7] "v"(xw[7]), [x8] "v"(xw[8]), [x9] "v"(xw[9]), [x10] "v"(xw[10]), [c0] "s"(c), [wr] "v"(wrow), [e] "v"(entry)
      : "v96", "v97", "v98", "v99", "v100", "v101", "v102", "v103", "v104", "v105", "v106", "v107", "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119", "v120", "v121", "v122", "v123", "v124", "v125", "v126", "v127", "v128", "v129", "v130", "v131", "v132", "v133", "v134", "v135", "v136", "v137", "v138", "v139", "v140", "v141", "v142", "v143", "v144", "v145", "v146", "v147", "v148", "v149", "v150", "v151", "v152", "v153", "v154", "v155", "v156", "v157", "v158", "v159", "v160", "v161", "v162", "v163", "v164", "v165", "v166", "v167", "v168", "v169", "v170", "v171", "v172", "v173", "v174", "v175", "v176", "v177", "v178", "v179", "v180", "v181", "v182", "v183", "v184", "v185", "v186", "v187", "v188", "v189", "v190", "v192", "v193", "v194", "v197", "v198", "memory");
}

struct V {
  static constexpr int NIN = 11, NACC = 12, NOUT = 12;
  static constexpr int kBatch = 4;
  static constexpr const int* kAccSlot = conv_e5m3_a4_o4::kAccSlot;
  static constexpr const int* kProdSlot = conv_e5m3_a4_o4::kProdSlot;
  static constexpr const int* kWSlot = conv_e5m3_a4_o4::kWSlot;
  static __device__ __forceinline__ void accum_batch(uint32_t (&acc)[(NACC + 3) & ~3],
                                                     const lds_u32* entry) {
    conv_e5m3_a4_o4::accum_batch(acc, entry);
  }
  static __device__ __forceinline__ void product_step(const uint32_t (&xw)[NIN], int c,
                                                      const lds_u32* wrow, lds_u32* entry) {
    conv_e5m3_a4_o4::product_step(xw, c, wrow, entry);
  }
  static __device__ __forceinline__ void product_batch(const uint32_t (&xw)[NIN], int c,
                                                       const lds_u32* wrow, lds_u32* entry) {
    conv_e5m3_a4_o4::product_batch(xw, c, wrow, entry);
  }
  static __device__ __forceinline__ void mac(uint32_t (&acc)[NACC], const uint32_t (&w)[NIN],
                                             const uint32_t (&x)[NIN]) { mac_e5m3_a4(acc, w, x); }
  static __device__ __forceinline__ void mul(const uint32_t (&w)[NIN], const uint32_t (&x)[NIN],
                                             uint32_t (&p)[NACC]) { prod_e5m3_a4(w, x, p); }
  static __device__ __forceinline__ void add(uint32_t (&acc)[NACC], const uint32_t (&p)[NACC]) {
    accum_e5m4(acc, p);
  }
  static __device__ __forceinline__ void epi(const uint32_t (&acc)[NACC], uint32_t (&out)[NOUT]) {
    epi_e5m4_o4(acc, out);
  }
};
}  // namespace conv_e5m3_a4_o4
hipError_t launch_conv_e5m3_a4_o4(const uint32_t* ifm, const uint32_t* w, uint32_t* ofm,
                              const ConvParams& p, int algo, hipStream_t stream) {
  dim3 grid((unsigned)((p.P + kConvBlock - 1) / kConvBlock), (unsigned)p.MT);
  if (algo == kAlgoSplit)
    hipLaunchKernelGGL(conv2d_split_kernel<conv_e5m3_a4_o4::V>, grid, dim3(2 * kConvBlock), 0, stream,
                       ifm, w, ofm, p);
  else
    hipLaunchKernelGGL(conv2d_kernel<conv_e5m3_a4_o4::V>, grid, dim3(kConvBlock), 0, stream, ifm, w, ofm, p);
  return hipGetLastError();
}
}  // namespace hobflops
