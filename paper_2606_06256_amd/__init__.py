"""SegPagedAttention with per-head page selection for AMD MI355X (gfx950).

The compute path is the C-ABI library libsegpa.so (hand-written HIP kernels);
`binding` is a thin ctypes layer over it and is imported on demand.
"""
