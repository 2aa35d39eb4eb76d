"""HCMS single-GPU hot path on MI355X (binding is added with the C ABI)."""
