"""MI355X-native region-wise multi-channel Winograd F(2x2,3x3) / F(4x4,3x3) convolution."""
