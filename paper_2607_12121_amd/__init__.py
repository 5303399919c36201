"""FlashDiff region-sparse DiT denoising step on MI355X (gfx950)."""
