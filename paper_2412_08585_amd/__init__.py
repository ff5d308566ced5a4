"""MI355X (gfx950) TurboAttention hot path: FlashQ + SAS quantized attention."""
