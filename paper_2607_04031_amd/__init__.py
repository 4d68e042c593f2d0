"""Tile-major GEMM for MI355X (gfx950): binding over the libtl C ABI."""
