"""MI355X-native 3D-RoPE + flash-attention forward (video-DiT attention hot path)."""
