"""MI355X-native W4A4 group-quantized GEMM (APEX4 hot path) -- Python binding."""
