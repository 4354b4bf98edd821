"""TRACK video-DiT denoiser hot path for MI355X."""
