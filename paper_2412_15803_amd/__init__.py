"""MI355X-native 4-bit group-quantized decode linears."""
