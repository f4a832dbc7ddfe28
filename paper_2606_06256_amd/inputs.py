"""Seeded synthetic inputs for SegPagedAttention workloads.

This module builds inputs only: random numbers, shapes, the segment and page
tables and the physical KV page pool. It contains none of the attention or
page-selection arithmetic. The CPU oracle and the GPU path both take their
inputs from here.

Every random value comes from a counter-based hash of (stream key, counter).
The hash is "lowbias32" (C. Wellons, hash-prospector, 2018), applied twice.
Normals come from the Box-Muller transform in float64, then round to float32
and then to bfloat16 (round to nearest even). The same torch code runs on CPU
or GPU, so a unit generated on the host for the oracle is bit-identical to the
copy written into the device pool. The tests check this on sampled units.

Pool layout (the contract of the fwd kernels; the header documents it too):
a physical page holds P tokens of ONE KV head, as P/16 tiles of 16 tokens.
  K tile: [D/8][16][8] bf16  (8-element chunks of the head dimension, chunk-major)
  V tile: [D][16]      bf16  (token-minor)
Slots past the context length inside the last page hold zeros.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from typing import Optional, Sequence

import numpy as np
import torch

TILE = 16  # tokens per tile; a page holds page_size / TILE tiles

_M32 = 0xFFFFFFFF

# stream kinds; each gets its own key space
KIND_Q, KIND_K, KIND_V, KIND_KSCALE, KIND_SHIFT_PAGE, KIND_SHIFT_DIR, KIND_PERM = 1, 2, 3, 4, 5, 6, 7
KIND_MASS = 8


def _lowbias32_int(x: int) -> int:
    x &= _M32
    x ^= x >> 16
    x = (x * 0x7FEB352D) & _M32
    x ^= x >> 15
    x = (x * 0x846CA68B) & _M32
    x ^= x >> 16
    return x


def stream_key(seed: int, kind: int, a: int = 0, b: int = 0) -> tuple[int, int]:
    """Two 32-bit keys for the stream (seed, kind, a, b)."""
    k1 = 0x243F6A88
    k2 = 0x85A308D3
    for v in (seed & _M32, (seed >> 32) & _M32, kind, a, b):
        k1 = _lowbias32_int(k1 ^ (v & _M32))
        k2 = _lowbias32_int(k2 ^ _lowbias32_int((v + 0x9E3779B9) & _M32))
    return k1, k2


def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    # (x * c) mod 2^32 for 0 <= x < 2^32 held in int64, without int64 overflow
    lo, hi = c & 0xFFFF, c >> 16
    return (x * lo + (((x * hi) & 0xFFFF) << 16)) & _M32


def _lowbias32(x: torch.Tensor) -> torch.Tensor:
    x = x ^ (x >> 16)
    x = _mul32(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32(x, 0x846CA68B)
    x = x ^ (x >> 16)
    return x


def hash_bits(key: tuple[int, int], counter: torch.Tensor) -> torch.Tensor:
    """32-bit hash of int64 counters in [0, 2^32) under a stream key."""
    return _lowbias32(_lowbias32(counter ^ key[0]) ^ key[1])


def normals_f64(key: tuple[int, int], start: int, count: int, device) -> torch.Tensor:
    """count N(0,1) draws (float64) for counters start .. start+count-1 (< 2^31)."""
    if start + count > (1 << 31):
        raise ValueError("counter range exceeds 2^31")
    idx = torch.arange(start, start + count, dtype=torch.int64, device=device)
    h1 = hash_bits(key, 2 * idx)
    h2 = hash_bits(key, 2 * idx + 1)
    u1 = (h1.to(torch.float64) + 0.5) * (1.0 / 4294967296.0)
    u2 = (h2.to(torch.float64) + 0.5) * (1.0 / 4294967296.0)
    return torch.sqrt(-2.0 * torch.log(u1)) * torch.cos((2.0 * math.pi) * u2)


def normals_np(key: tuple[int, int], count: int) -> np.ndarray:
    return normals_f64(key, 0, count, "cpu").numpy()


def to_bf16(x64: torch.Tensor) -> torch.Tensor:
    """float64 -> float32 -> bfloat16, each step round-to-nearest-even."""
    return x64.to(torch.float32).to(torch.bfloat16)


# --------------------------------------------------------------------------
# workload description
# --------------------------------------------------------------------------
SEL_ALL, SEL_HEAD_CLASS, SEL_RANDOM_HASH, SEL_TOPK_MEANKEY = 0, 1, 2, 3


@dataclass
class Spec:
    name: str
    B: int
    Hq: int
    Hkv: int
    D: int
    P: int                      # page size (tokens), multiple of 16
    seg_tokens: int             # segment length (tokens), multiple of P
    ctx_lens: Sequence[int]     # KV length per request, including the query chunk
    q_lens: Sequence[int]       # query tokens per request
    seed: int
    sel_mode: int = SEL_ALL
    budgets: Optional[Sequence[int]] = None  # selected-page budget per request
    forced_head: int = 0        # always-selected leading pages
    forced_tail: int = 0        # always-selected trailing pages
    sel_seed: int = 0           # RANDOM_HASH seed
    n_sink: int = 4             # HEAD_CLASS sink tokens
    window: int = 256           # HEAD_CLASS window w
    head_policy: Optional[Sequence[int]] = None  # per KV head, 1 = global, 0 = local
    k_page_scale_sigma: float = 0.0  # > 0: K of each page scaled by LogNormal(0, sigma)
    shift_pages: int = 0        # per unit: this many pages get +shift_mag * u on every key
    shift_mag: float = 0.0
    extra_phys_pages: int = 0   # unused physical pages appended to the pool
    shared_prefix_segments: int = 0  # requests r > 0 alias request 0's first segments
    description: str = ""


def cdiv(a: int, b: int) -> int:
    return -(-a // b)


@dataclass
class Workload:
    spec: Spec
    ctx_lens: np.ndarray        # int32 [B]
    q_indptr: np.ndarray        # int32 [B+1]
    n_pages: np.ndarray         # int64 [B]
    budgets: np.ndarray         # int32 [B]
    seg_table: np.ndarray       # int32 [B, Hkv, max_segments]
    page_table: np.ndarray      # int32 [num_virtual]
    num_phys: int
    page_valid: np.ndarray      # int32 [num_phys] valid tokens per physical page
    vbase: np.ndarray           # int64 [B, Hkv] first virtual page of each unit (owned pages)
    head_policy: np.ndarray     # int8 [Hkv]
    _kscale_cache: dict = field(default_factory=dict)

    # ---- shape helpers -------------------------------------------------
    @property
    def B(self): return self.spec.B
    @property
    def Hq(self): return self.spec.Hq
    @property
    def Hkv(self): return self.spec.Hkv
    @property
    def G(self): return self.spec.Hq // self.spec.Hkv
    @property
    def D(self): return self.spec.D
    @property
    def P(self): return self.spec.P
    @property
    def pps(self): return self.spec.seg_tokens // self.spec.P
    @property
    def max_segments(self): return self.seg_table.shape[2]
    @property
    def total_q(self): return int(self.q_indptr[-1])
    @property
    def num_units(self): return self.B * self.Hkv
    @property
    def max_q_len(self): return int(np.max(np.diff(self.q_indptr))) if self.B else 0

    # ---- logical data --------------------------------------------------
    def q(self, device="cpu") -> torch.Tensor:
        n = self.total_q * self.Hq * self.D
        z = normals_f64(stream_key(self.spec.seed, KIND_Q), 0, n, device)
        return to_bf16(z).reshape(self.total_q, self.Hq, self.D)

    def _kscale(self, r: int, g: int) -> Optional[np.ndarray]:
        sp = self.spec
        if sp.k_page_scale_sigma <= 0:
            return None
        key = (r, g)
        if key not in self._kscale_cache:
            n = int(self.n_pages[r])
            z = normals_np(stream_key(sp.seed, KIND_KSCALE, r, g), n)
            self._kscale_cache[key] = np.exp(sp.k_page_scale_sigma * z)
        return self._kscale_cache[key]

    def shifted_pages(self, r: int, g: int) -> np.ndarray:
        """Logical pages of unit (r, g) whose keys get the mean shift."""
        sp = self.spec
        n = int(self.n_pages[r])
        m = min(sp.shift_pages, n)
        if m <= 0:
            return np.zeros(0, dtype=np.int64)
        key = stream_key(sp.seed, KIND_SHIFT_PAGE, r, g)
        h = hash_bits(key, torch.arange(n, dtype=torch.int64)).numpy()
        order = np.lexsort((np.arange(n), h))
        return np.sort(order[:m])

    def shift_vector(self) -> np.ndarray:
        """shift_mag * u with u a seeded unit vector in R^D (float64)."""
        sp = self.spec
        z = normals_np(stream_key(sp.seed, KIND_SHIFT_DIR), sp.D)
        return sp.shift_mag * (z / np.sqrt(np.sum(z * z)))

    def _unit_stream(self, r: int, g: int, kind: int, L: int, device) -> torch.Tensor:
        """float64 [L, D] draws of unit (r, g), honouring prefix aliasing."""
        sp = self.spec
        D = sp.D
        shared = min(L, sp.shared_prefix_segments * sp.seg_tokens) if r > 0 else 0
        parts = []
        if shared > 0:
            parts.append(normals_f64(stream_key(sp.seed, kind, 0, g), 0, shared * D, device))
        if L > shared:
            parts.append(normals_f64(stream_key(sp.seed, kind, r, g), shared * D, (L - shared) * D, device))
        z = torch.cat(parts) if len(parts) > 1 else parts[0]
        return z.reshape(L, D)

    def unit_kv(self, r: int, g: int, device="cpu") -> tuple[torch.Tensor, torch.Tensor]:
        """Logical K, V of unit (r, g): bf16 [L, D] each (token-major)."""
        sp = self.spec
        L = int(self.ctx_lens[r])
        if L == 0:
            e = torch.zeros(0, sp.D, dtype=torch.bfloat16, device=device)
            return e, e.clone()
        zk = self._unit_stream(r, g, KIND_K, L, device)
        zv = self._unit_stream(r, g, KIND_V, L, device)
        scale = self._kscale(r, g)
        if scale is not None:
            s_tok = np.repeat(scale, sp.P)[:L]
            zk = zk * torch.from_numpy(s_tok).to(device=device, dtype=torch.float64)[:, None]
        if sp.shift_pages > 0:
            pages = self.shifted_pages(r, g)
            if len(pages):
                tok = (pages[:, None] * sp.P + np.arange(sp.P)[None, :]).reshape(-1)
                tok = tok[tok < L]
                sv = torch.from_numpy(self.shift_vector()).to(device)
                ti = torch.from_numpy(tok).to(device)
                zk[ti] = zk[ti] + sv[None, :]
        return to_bf16(zk), to_bf16(zv)

    # ---- physical pool -------------------------------------------------
    def unit_phys_pages(self, r: int, g: int) -> np.ndarray:
        """Physical page of each logical page of unit (r, g), via the tables."""
        n = int(self.n_pages[r])
        j = np.arange(n)
        seg = self.seg_table[r, g, j // self.pps]
        return self.page_table[seg + j % self.pps]

    def tile_unit(self, K: torch.Tensor, V: torch.Tensor, n_pages: int):
        """Logical [L, D] K/V -> pool page images [n_pages, P*D] in the tile layout."""
        P, D = self.P, self.D
        L = K.shape[0]
        pad = n_pages * P - L
        if pad:
            K = torch.cat([K, torch.zeros(pad, D, dtype=K.dtype, device=K.device)])
            V = torch.cat([V, torch.zeros(pad, D, dtype=V.dtype, device=V.device)])
        nt = n_pages * (P // TILE)
        kt = K.reshape(nt, TILE, D // 8, 8).permute(0, 2, 1, 3).contiguous()
        vt = V.reshape(nt, TILE, D).permute(0, 2, 1).contiguous()
        return kt.reshape(n_pages, P * D), vt.reshape(n_pages, P * D)

    def build_pool(self, device="cpu") -> tuple[torch.Tensor, torch.Tensor]:
        """Physical K and V pools, bf16 [num_phys, P*D], written unit by unit."""
        P, D = self.P, self.D
        kp = torch.zeros(self.num_phys, P * D, dtype=torch.bfloat16, device=device)
        vp = torch.zeros(self.num_phys, P * D, dtype=torch.bfloat16, device=device)
        for r in range(self.B):
            n = int(self.n_pages[r])
            if n == 0:
                continue
            for g in range(self.Hkv):
                K, V = self.unit_kv(r, g, device)
                kt, vt = self.tile_unit(K, V, n)
                phys = torch.from_numpy(self.unit_phys_pages(r, g).astype(np.int64)).to(device)
                kp[phys] = kt
                vp[phys] = vt
                del K, V, kt, vt
        return kp, vp

    # ---- bookkeeping for measurement -----------------------------------
    def attended_tokens(self, sel_indptr: np.ndarray, sel_pages: np.ndarray) -> int:
        """Sum over units of selected valid tokens (a count, not a result)."""
        tot = 0
        P = self.P
        for u in range(self.num_units):
            r = u // self.Hkv
            L = int(self.ctx_lens[r])
            pg = sel_pages[sel_indptr[u]:sel_indptr[u + 1]].astype(np.int64)
            tot += int(np.sum(np.minimum(P, L - pg * P)))
        return tot


def build(spec: Spec) -> Workload:
    """Derive tables and bookkeeping from a Spec (host side, deterministic)."""
    sp = spec
    if sp.Hq % sp.Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    if sp.shared_prefix_segments and (sp.k_page_scale_sigma > 0 or sp.shift_pages):
        raise ValueError("prefix aliasing is not combined with per-page K scaling or shifts")
    if sp.P % TILE or sp.seg_tokens % sp.P or sp.D % 8:
        raise ValueError("page size must be a multiple of 16 and divide the segment length")
    B, Hkv, P = sp.B, sp.Hkv, sp.P
    pps = sp.seg_tokens // P
    ctx = np.asarray(sp.ctx_lens, dtype=np.int64)
    ql = np.asarray(sp.q_lens, dtype=np.int64)
    assert ctx.shape == (B,) and ql.shape == (B,)
    if np.any(ql > ctx):
        raise ValueError("query chunk longer than the context")
    n_pages = (ctx + P - 1) // P
    nseg = (n_pages + pps - 1) // pps
    max_segments = max(1, int(nseg.max()) if B else 1)
    seg_table = np.full((B, Hkv, max_segments), -1, dtype=np.int64)
    vbase = np.zeros((B, Hkv), dtype=np.int64)
    nv = 0
    shared = sp.shared_prefix_segments
    for r in range(B):
        for g in range(Hkv):
            vbase[r, g] = nv
            for s in range(int(nseg[r])):
                if r > 0 and s < shared and s < int(nseg[0]):
                    seg_table[r, g, s] = seg_table[0, g, s]
                else:
                    seg_table[r, g, s] = nv
                    nv += pps
    num_virtual = nv
    num_phys = num_virtual + sp.extra_phys_pages
    # physical placement: a seeded random injection of virtual pages into the pool
    perm_key = stream_key(sp.seed, KIND_PERM)
    h = hash_bits(perm_key, torch.arange(num_phys, dtype=torch.int64)).numpy()
    order = np.lexsort((np.arange(num_phys), h))
    page_table = order[:num_virtual].astype(np.int64)
    # valid tokens of every physical page (0 for unused pages)
    page_valid = np.zeros(num_phys, dtype=np.int64)
    for r in range(B):
        j = np.arange(int(n_pages[r]))
        valid = np.minimum(P, int(ctx[r]) - j * P)
        for g in range(Hkv):
            page_valid[page_table[seg_table[r, g, j // pps] + j % pps]] = valid
    if sp.budgets is None:
        budgets = n_pages.copy()
    else:
        budgets = np.asarray(sp.budgets, dtype=np.int64)
    hp = np.asarray(sp.head_policy if sp.head_policy is not None else [1] * Hkv, dtype=np.int8)
    q_indptr = np.concatenate([[0], np.cumsum(ql)]).astype(np.int32)
    return Workload(spec=sp, ctx_lens=ctx.astype(np.int32), q_indptr=q_indptr,
                    n_pages=n_pages, budgets=budgets.astype(np.int32),
                    seg_table=seg_table.astype(np.int32), page_table=page_table.astype(np.int32),
                    num_phys=num_phys, page_valid=page_valid.astype(np.int32), vbase=vbase,
                    head_policy=hp)


# --------------------------------------------------------------------------
# the five named workloads
# --------------------------------------------------------------------------
def config_spec(i: int) -> Spec:
    """Named workloads 1..10 (shapes of the paper's Llama/Qwen-style layers;
    6..9 are the head-class micro-benchmark shape of Section 5.3; 10 is
    workload 2 as multi-head attention)."""
    seed = 1000 + i
    if i == 1:
        return Spec(name="tiny", B=1, Hq=4, Hkv=4, D=64, P=16, seg_tokens=256,
                    ctx_lens=[1024], q_lens=[1], seed=seed, sel_mode=SEL_ALL,
                    description="1 request, 4/4 heads, D64, 1 decode token, 1024 tokens "
                                "= 4 segments x 256, page 16, all pages")
    if i == 2:
        n = 32768 // 16
        return Spec(name="llama3_8b_decode", B=16, Hq=32, Hkv=8, D=128, P=16, seg_tokens=2048,
                    ctx_lens=[32768] * 16, q_lens=[1] * 16, seed=seed, sel_mode=SEL_RANDOM_HASH,
                    budgets=[cdiv(n, 4)] * 16, forced_head=2048 // 16, forced_tail=2048 // 16,
                    sel_seed=0x5E6A11, description="batch 16, 32/8 heads, D128, 32K context "
                    "in 2048-token segments, page 16, 25% of pages incl. first+last segment")
    if i == 3:
        rng = np.random.default_rng(seed)
        L = np.floor(np.exp(rng.uniform(math.log(4096), math.log(131072), size=64))).astype(np.int64)
        beta = rng.uniform(0.05, 0.50, size=64)
        npg = (L + 15) // 16
        budgets = [int(math.ceil(b * n)) for b, n in zip(beta, npg)]
        return Spec(name="varlen_sparse_decode", B=64, Hq=32, Hkv=8, D=128, P=16, seg_tokens=4096,
                    ctx_lens=L.tolist(), q_lens=[1] * 64, seed=seed, sel_mode=SEL_RANDOM_HASH,
                    budgets=budgets, sel_seed=0x5E6A13, k_page_scale_sigma=0.5,
                    description="batch 64, 32/8 heads, D128, context log-uniform in "
                    "[4096, 131072], segment 4096, page 16, budget U[5%,50%], "
                    "K page scale LogNormal(0, 0.5)")
    if i == 4:
        prior, chunk = 65536, 512
        return Spec(name="chunked_prefill", B=4, Hq=32, Hkv=8, D=128, P=16, seg_tokens=4096,
                    ctx_lens=[prior + chunk] * 4, q_lens=[chunk] * 4, seed=seed,
                    sel_mode=SEL_RANDOM_HASH, budgets=[cdiv(prior // 16 * 20, 100) + chunk // 16] * 4,
                    forced_tail=chunk // 16, sel_seed=0x5E6A14,
                    description="batch 4, 512-token causal chunk, 32/8 heads, D128, 64K prior "
                    "context in 4096-token segments, page 16, 20% of prior pages + chunk pages")
    if i == 5:
        n = 131072 // 32
        return Spec(name="select_attend", B=32, Hq=64, Hkv=8, D=128, P=32, seg_tokens=8192,
                    ctx_lens=[131072] * 32, q_lens=[1] * 32, seed=seed, sel_mode=SEL_TOPK_MEANKEY,
                    budgets=[cdiv(n, 10)] * 32, shift_pages=cdiv(2 * n, 100), shift_mag=3.0,
                    description="batch 32 decode, 64/8 heads, D128, 128K context, segment 8192, "
                    "page 32, top-10% pages by (sum of group queries) . mean key; 2% of pages "
                    "shifted by +3 along a seeded direction")
    if i in (6, 7, 8):
        return headclass_spec(i, {6: 8192, 7: 32768, 8: 131072}[i], q_len=1)
    if i == 10:
        # workload 2 with one query head per KV head (multi-head attention):
        # a decode tile then fills one row of the 16-row matrix-core tile
        n = 32768 // 16
        return Spec(name="mha_decode", B=16, Hq=32, Hkv=32, D=128, P=16, seg_tokens=2048,
                    ctx_lens=[32768] * 16, q_lens=[1] * 16, seed=seed, sel_mode=SEL_RANDOM_HASH,
                    budgets=[cdiv(n, 4)] * 16, forced_head=2048 // 16, forced_tail=2048 // 16,
                    sel_seed=0x5E6A1A, description="batch 16, 32/32 heads (MHA), D128, 32K "
                    "context in 2048-token segments, page 16, 25% of pages incl. first+last segment")
    if i == 9:
        return headclass_spec(i, 32768, q_len=512)
    raise ValueError(f"no workload {i}")


def headclass_spec(i: int, ctx: int, q_len: int, layers: int = 64) -> Spec:
    """The paper's own micro-benchmark shape: Qwen3-32B-like layers (32/8
    heads, D128), half of the KV heads global (all pages) and half local
    (4 sink tokens + a 316-token window: a 320-token window), run for 64
    layers as one batched call (each layer is one request of the batch: its
    own segment table rows and pages)."""
    kind = "decode" if q_len == 1 else f"prefill of a {q_len}-token chunk"
    return Spec(name=f"qwen3_32b_headclass_{'decode' if q_len == 1 else 'prefill'}_{ctx // 1024}k",
                B=layers, Hq=32, Hkv=8, D=128, P=16, seg_tokens=2048,
                ctx_lens=[ctx] * layers, q_lens=[q_len] * layers, seed=1000 + i,
                sel_mode=SEL_HEAD_CLASS, head_policy=[1, 0] * 4, n_sink=4, window=316,
                description=f"{layers} layers x 1 request (one batched call), 32/8 heads, D128, "
                            f"{ctx // 1024}K context in 2048-token segments, page 16, {kind}; "
                            f"KV heads alternate global (all pages) / local (sink 4 + window 316)")


def config(i: int) -> Workload:
    return build(config_spec(i))


def scaled_spec(i: int, ctx_div: int = 1, batch: Optional[int] = None) -> Spec:
    """A smaller copy of workload i (same structure) for quick checks."""
    sp = config_spec(i)
    B = batch if batch is not None else sp.B
    ctx = [max(1, int(c) // ctx_div) for c in list(sp.ctx_lens)[:B]]
    ql = [min(q, c) for q, c in zip(list(sp.q_lens)[:B], ctx)]
    seg = max(sp.P, sp.seg_tokens // ctx_div)
    seg -= seg % sp.P
    npg = [cdiv(c, sp.P) for c in ctx]
    if sp.budgets is not None:
        fr = [b / cdiv(int(c0), sp.P) for b, c0 in zip(list(sp.budgets)[:B], list(sp.ctx_lens)[:B])]
        budgets = [max(1, int(math.ceil(f * n))) for f, n in zip(fr, npg)]
    else:
        budgets = None
    fh = sp.forced_head // ctx_div if sp.forced_head else 0
    ft = sp.forced_tail // ctx_div if sp.forced_tail else 0
    if i == 4:
        ft = cdiv(ql[0], sp.P)
    return replace(sp, name=sp.name + f"_div{ctx_div}", B=B, ctx_lens=ctx, q_lens=ql,
                   seg_tokens=seg, budgets=budgets, forced_head=fh, forced_tail=ft,
                   shift_pages=cdiv(sp.shift_pages, ctx_div) if sp.shift_pages else 0)


# --------------------------------------------------------------------------
# synthetic per-token attention masses (inputs of the token selection)
# --------------------------------------------------------------------------
def synthetic_masses(seed: int, rows: int, cols: int, kind: str = "lognormal") -> np.ndarray:
    """float32 [rows, cols] of nonnegative per-(token, head) masses.

    lognormal: exp(2.5 * N(0,1)) / cols, a heavy tail like the attention mass
      of long chunks, where a small fraction of tokens carries most of it;
    dyadic: multiples of 2^-10 below 1/16 (many equal values; every float64
      partial sum is exact);
    sparse: 0 for about 90% of the entries, lognormal for the rest.
    """
    key = stream_key(seed, KIND_MASS, cols, {"lognormal": 0, "dyadic": 1, "sparse": 2}[kind])
    n = rows * cols
    if kind == "dyadic":
        h = hash_bits(key, torch.arange(n, dtype=torch.int64)).numpy()
        return ((h % 64).astype(np.float64) * 2.0 ** -10).astype(np.float32).reshape(rows, cols)
    z = normals_np(key, n)
    m = np.exp(2.5 * z) / cols
    if kind == "sparse":
        h = hash_bits(stream_key(seed, KIND_MASS, cols, 3), torch.arange(n, dtype=torch.int64)).numpy()
        m = np.where(h % 10 == 0, m, 0.0)
    return m.astype(np.float32).reshape(rows, cols)
