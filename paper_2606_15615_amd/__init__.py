"""MI355X-native branch-cached DiT-MoE layer step (MoECa)."""
