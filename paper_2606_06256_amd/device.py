"""Device-resident copy of a synthetic workload, driving the C-ABI calls.

Memory plumbing only: torch allocates the device buffers, and the binding
passes their pointers to libsegpa.so. One `step()` is one pass of the hot
path: page selection (plus, for TOPK_MEANKEY, the scoring pass over the page
key sums) and the attention forward with its split combine.
"""
from __future__ import annotations

import numpy as np
import torch

from . import binding as B
from . import inputs as I


class DeviceWorkload:
    def __init__(self, wl: I.Workload, device: str = "cuda", build_pool: bool = True):
        self.wl = wl
        sp = wl.spec
        self.device = device
        dev = torch.device(device)
        self.mode = sp.sel_mode
        self.q = wl.q(dev)
        self.q_indptr = torch.from_numpy(wl.q_indptr.astype(np.int32)).to(dev)
        self.ctx_lens = torch.from_numpy(wl.ctx_lens.astype(np.int32)).to(dev)
        self.seg_table = torch.from_numpy(wl.seg_table.reshape(-1).astype(np.int32)).to(dev)
        self.page_table = torch.from_numpy(wl.page_table.astype(np.int32)).to(dev)
        if self.page_table.numel() == 0:
            self.page_table = torch.zeros(1, dtype=torch.int32, device=dev)
        self.budgets = torch.from_numpy(wl.budgets.astype(np.int32)).to(dev)
        self.head_policy = torch.from_numpy(wl.head_policy.astype(np.int8)).to(dev)
        self.page_valid = torch.from_numpy(wl.page_valid.astype(np.int32)).to(dev)
        if build_pool:
            self.k_pool, self.v_pool = wl.build_pool(dev)
        self.dims = B.make_dims(num_requests=wl.B, num_q_heads=wl.Hq, num_kv_heads=wl.Hkv,
                                head_dim=wl.D, page_size=wl.P, pages_per_segment=wl.pps,
                                max_segments=wl.max_segments, max_q_len=max(1, wl.max_q_len),
                                total_q=wl.total_q, num_virtual_pages=int(wl.page_table.size),
                                num_phys_pages=int(wl.num_phys))
        self.capacity = wl.num_units * wl.max_segments * wl.pps
        self.sel_indptr = torch.zeros(wl.num_units + 1, dtype=torch.int32, device=dev)
        self.sel_pages = torch.zeros(max(1, self.capacity), dtype=torch.int32, device=dev)
        self.out = torch.zeros(max(1, wl.total_q), wl.Hq, wl.D, dtype=torch.bfloat16, device=dev)
        self.lse = torch.zeros(max(1, wl.total_q), wl.Hq, dtype=torch.float32, device=dev)
        ws = B.seg_paged_attn_workspace_size(self.dims, self.mode)
        if ws <= 0:
            raise RuntimeError("seg_paged_attn_workspace_size rejected the dimensions")
        self.workspace = torch.zeros(ws, dtype=torch.uint8, device=dev)
        self.page_ksum = None
        if self.mode == I.SEL_TOPK_MEANKEY:
            self.page_ksum = torch.zeros(wl.num_phys, wl.D, dtype=torch.float32, device=dev)
        self.params = B.make_select_params(
            self.mode, n_sink_tokens=sp.n_sink, window_tokens=sp.window,
            forced_head_pages=sp.forced_head, forced_tail_pages=sp.forced_tail, seed=sp.sel_seed,
            head_policy=self.head_policy, budget_pages=self.budgets)

    # ---- the C-ABI calls ------------------------------------------------
    def summary(self, stream=None):
        B.seg_paged_attn_page_summary(self.dims, self.k_pool, self.page_valid, self.page_ksum, stream)

    def select(self, stream=None):
        B.seg_paged_attn_select(self.dims, self.params, self.ctx_lens, self.q, self.q_indptr,
                                self.page_ksum, self.seg_table, self.page_table, self.sel_indptr,
                                self.sel_pages, self.workspace, stream)

    def fwd(self, stream=None, sel_indptr=None, sel_pages=None):
        B.seg_paged_attn_fwd(self.dims, self.q, self.q_indptr, self.ctx_lens, self.k_pool,
                             self.v_pool, self.seg_table, self.page_table,
                             self.sel_indptr if sel_indptr is None else sel_indptr,
                             self.sel_pages if sel_pages is None else sel_pages,
                             self.out, self.lse, self.workspace, stream)

    def token_mass(self, stream=None):
        """Mass of every chunk token per KV head, from the last fwd's lse."""
        if getattr(self, "mass", None) is None:
            self.mass = torch.zeros(max(1, self.wl.total_q), self.wl.Hkv, dtype=torch.float32,
                                    device=self.device)
        B.seg_paged_attn_token_mass(self.dims, self.q, self.q_indptr, self.ctx_lens, self.k_pool,
                                    self.seg_table, self.page_table, self.sel_indptr,
                                    self.sel_pages, self.lse, self.mass, stream)

    def select_tokens(self, tau: float, recent: int, stream=None):
        """Tokens kept by cumulative mass (needs token_mass() first)."""
        if getattr(self, "keep", None) is None:
            n = max(1, self.wl.total_q)
            self.keep = torch.zeros(n, dtype=torch.uint8, device=self.device)
            self.kept = torch.zeros(n, dtype=torch.int32, device=self.device)
            self.keep_count = torch.zeros(self.wl.B, dtype=torch.int32, device=self.device)
            self.tok_mass = torch.zeros(n, dtype=torch.float32, device=self.device)
        B.seg_paged_attn_select_tokens(self.dims, self.q_indptr, self.mass, tau, recent, self.keep,
                                       self.keep_count, self.kept, self.tok_mass, stream)

    def step(self, stream=None):
        self.select(stream)
        self.fwd(stream)

    def validate(self, stream=None):
        return B.seg_paged_attn_validate(self.dims, self.ctx_lens, self.q_indptr, self.seg_table,
                                         self.page_table, self.sel_indptr, self.sel_pages,
                                         self.workspace, stream)

    # ---- host copies of results -----------------------------------------
    def selection(self):
        ind = self.sel_indptr.cpu().numpy().astype(np.int64)
        pages = self.sel_pages[: max(1, int(ind[-1]))].cpu().numpy()
        return ind, pages

    def set_selection(self, lists):
        """Upload explicit per-unit page lists (ascending logical ids)."""
        ind = np.zeros(self.wl.num_units + 1, dtype=np.int64)
        for u, p in enumerate(lists):
            ind[u + 1] = ind[u] + len(p)
        flat = np.concatenate([np.asarray(p, dtype=np.int32) for p in lists]) if ind[-1] else np.zeros(0, np.int32)
        self.sel_indptr.copy_(torch.from_numpy(ind.astype(np.int32)))
        self.sel_pages.zero_()
        if len(flat):
            self.sel_pages[: len(flat)].copy_(torch.from_numpy(flat))
