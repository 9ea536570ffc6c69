"""MI355X-native BFLA block-filtered sparse causal prefill (HIP, gfx950)."""
