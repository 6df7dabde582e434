"""MI355X-native block-sparse attention with a reusable block mask (Chorus II hot path)."""
