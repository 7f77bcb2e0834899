"""HOBFLOPS on MI355X: bitsliced custom-precision floating-point MCMK convolution."""
