"""seg_paged_attn_fwd_noalloc (the forward over the library's built-in
per-GPU scratch, for callers that cannot allocate) against
seg_paged_attn_fwd with a caller workspace: the same kernels, so the outputs
must agree bit for bit, and both must meet the oracle's tolerance. Two calls
in a row on the shared scratch, the second with a smaller input, then a
chunked prefill (no partials) and a shape whose partials exceed the scratch
(refused before any launch)."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2606_06256_amd import binding as B
from paper_2606_06256_amd import inputs as I
from paper_2606_06256_amd.device import DeviceWorkload

import parity_util as PU

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.detach().contiguous().view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).cpu()


def _noalloc_matches_fwd(wl, label):
    print(f"[no_alloc] {label}: B={wl.B} Hq={wl.Hq} Hkv={wl.Hkv} D={wl.D} P={wl.P}", flush=True)
    dw = DeviceWorkload(wl)
    if wl.spec.sel_mode == I.SEL_TOPK_MEANKEY:
        dw.summary()
    dw.select()
    dw.fwd()
    torch.cuda.synchronize()
    ref_out, ref_lse = dw.out.clone(), dw.lse.clone()
    dw.out.fill_(7.0)                      # every output must be rewritten
    dw.lse.fill_(123.0)
    B.seg_paged_attn_fwd_noalloc(dw.dims, dw.q, dw.q_indptr, dw.ctx_lens, dw.k_pool, dw.v_pool,
                                 dw.seg_table, dw.page_table, dw.sel_indptr, dw.sel_pages, dw.out,
                                 dw.lse)
    torch.cuda.synchronize()
    assert torch.equal(_bits(dw.out), _bits(ref_out)), f"{label}: output differs from fwd"
    assert torch.equal(_bits(dw.lse), _bits(ref_lse)), f"{label}: lse differs from fwd"
    q64 = wl.q("cpu").double().numpy()
    units = PU.sample_units(wl.num_units, 4)
    want = PU.oracle_selection(wl, q64, units=units)
    stats = PU.compare_outputs(wl, dw, q64, want, units)
    print(f"[no_alloc] {label}: {stats}", flush=True)
    stats.check(label)
    return dw


def test_noalloc_two_calls_then_smaller_input():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    # 16 units x 128 selected pages: every unit spans several waves (split partials)
    _noalloc_matches_fwd(I.build(I.scaled_spec(2, 4, 4)), "llama3-decode/4")
    # a smaller input on the same scratch: the earlier call's partials must not leak in
    _noalloc_matches_fwd(I.build(I.scaled_spec(3, 32, 3)), "varlen-decode/32")
    _noalloc_matches_fwd(I.config(1), "tiny")


def test_noalloc_chunked_prefill_and_topk():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    sp = I.scaled_spec(4, 32, 2)
    sp.q_lens = [48, 31]
    sp.ctx_lens = [2048 + 48, 1500 + 31]
    sp.budgets = [40, 30]
    _noalloc_matches_fwd(I.build(sp), "prefill")
    _noalloc_matches_fwd(I.build(I.scaled_spec(5, 32, 2)), "topk-decode/32")


def test_noalloc_refuses_partials_beyond_its_scratch():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    # 8192 units x 8 row blocks of decode partials: far beyond the scratch;
    # refused by the host check, nothing launched (the pointers are never read)
    dims = B.make_dims(num_requests=1024, num_q_heads=64, num_kv_heads=8, head_dim=128, page_size=16,
                       pages_per_segment=4, max_segments=4, max_q_len=15, total_q=1024 * 15,
                       num_virtual_pages=64, num_phys_pages=64)
    assert B.seg_paged_attn_workspace_size(dims, 0) > B.SPA_NOALLOC_SCRATCH_BYTES
    fake = ctypes.c_void_p(0x1000)
    st = B.lib().seg_paged_attn_fwd_noalloc(ctypes.byref(dims), fake, fake, fake, fake, fake, fake,
                                            fake, fake, fake, 1 << 20, fake, None, None)
    assert st == B.SPA_ERR_WORKSPACE
