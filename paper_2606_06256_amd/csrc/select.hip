// Page selection (SelectVisibleState): per-unit logical page lists as CSR.
//
// ALL and HEAD_CLASS follow the policy step of Algorithm 2 (a global head
// keeps its full page range; a local head keeps the pages that overlap the sink
// tokens or the window W(i) = S_sink U [max(0, i - w), i] of Section 4.2 of any
// query of the chunk; Section 4.3: whole overlapping pages). RANDOM_HASH and
// TOPK_MEANKEY rank the non-forced pages by a 64-bit key (SplitMix64 hash, or
// the order-preserving image of the float64 mean-key score) and keep the
// `budget - forced` smallest keys, equal keys to the lower page index.
//
// One block per unit. Every count is a closed-form function of the context
// length, the query count and the parameters, so each block derives its CSR
// offset by summing the counts of the units before it: no second launch and
// no device-wide synchronisation. The ranked rules find the exact threshold
// key by an 8-pass radix select (8-bit digits, LDS histogram) and then emit the
// chosen pages in ascending order with block-wide prefix counts.
#include "common.hpp"
#include "kernels.hpp"

namespace segpa {

namespace {

constexpr int kModeAll = 0, kModeHeadClass = 1, kModeRandom = 2, kModeTopk = 3;

struct UnitInfo {
  int n;        // logical pages
  int count;    // selected pages
  int a_end;    // HEAD_CLASS: sink pages [0, a_end); ranked: forced head [0, a_end)
  int b_begin;  // HEAD_CLASS: window pages [b_begin, n); ranked: forced tail [b_begin, n)
};

__device__ UnitInfo unit_info(const SelArgs& a, int u) {
  const int r = u / a.Hkv;
  const int g = u - r * a.Hkv;
  const int max_tokens = a.max_segs * a.pps * a.P;
  const int L = clampv(a.ctx_lens[r], 0, max_tokens);
  UnitInfo I;
  I.n = (L + a.P - 1) / a.P;
  I.count = I.n;
  I.a_end = I.n;
  I.b_begin = I.n;
  if (a.mode == kModeHeadClass) {
    if (a.head_policy[g] == 0) {   // local head
      const int nq = a.q_indptr != nullptr ? clampv(a.q_indptr[r + 1] - a.q_indptr[r], 0, L) : 1;
      const int ns = clampv(a.n_sink, 0, L);
      const int sinkp = min(I.n, (ns + a.P - 1) / a.P);
      const int winlo = nq > 0 ? min(I.n, max(0, L - nq - a.window) / a.P) : I.n;
      I.a_end = sinkp;
      I.b_begin = winlo;
      I.count = winlo <= sinkp ? I.n : sinkp + (I.n - winlo);
      if (winlo <= sinkp) { I.a_end = I.n; I.b_begin = I.n; }
    }
  } else if (a.mode == kModeRandom || a.mode == kModeTopk) {
    const int fh = min(I.n, a.forced_head);
    const int ft = min(I.n, a.forced_tail);
    const int forced = min(I.n, fh + ft);
    const int b = max(0, a.budget[r]);
    I.a_end = fh;
    I.b_begin = max(fh, I.n - ft);
    I.count = min(I.n, max(b, forced));
  }
  return I;
}

__device__ __forceinline__ uint64_t random_key(uint64_t sm_seed, int r, int g, int p) {
  return splitmix64(sm_seed ^ (((uint64_t)r << 40) | ((uint64_t)g << 32) | (uint32_t)p));
}

// Order-preserving map of a float64 score such that higher scores give smaller
// keys; -0 equals +0; NaN ranks after every number.
__device__ __forceinline__ uint64_t descending_key(double s) {
  if (s != s) return ~0ull;
  if (s == 0.0) s = 0.0;
  const uint64_t b = (uint64_t)__double_as_longlong(s);
  const uint64_t ascending = (b >> 63) ? ~b : (b | 0x8000000000000000ull);
  return ~ascending;
}

template <int BS>
__device__ int64_t block_sum64(int64_t v, int64_t* scratch) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) scratch[w] = v;
  __syncthreads();
  int64_t t = 0;
#pragma unroll
  for (int i = 0; i < BS / 64; ++i) t += scratch[i];
  __syncthreads();
  return t;
}

// Block-wide exclusive prefix counts of two predicates, in thread order, and
// their block totals.
template <int BS>
__device__ void block_scan2(bool x, bool y, int& ex_x, int& ex_y, int& tot_x, int& tot_y,
                            int* scratch) {
  const uint64_t bx = __ballot(x);
  const uint64_t by = __ballot(y);
  const int w = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  if (lane == 0) {
    scratch[w] = __popcll(bx);
    scratch[BS / 64 + w] = __popcll(by);
  }
  __syncthreads();
  int px = 0, py = 0;
  tot_x = 0;
  tot_y = 0;
#pragma unroll
  for (int i = 0; i < BS / 64; ++i) {
    const int cx = scratch[i], cy = scratch[BS / 64 + i];
    if (i < w) { px += cx; py += cy; }
    tot_x += cx;
    tot_y += cy;
  }
  ex_x = px + lane_prefix_count(bx);
  ex_y = py + lane_prefix_count(by);
  __syncthreads();
}

}  // namespace

__global__ __launch_bounds__(kSelectBlock) void select_fill_kernel(const SelArgs a) {
  constexpr int BS = kSelectBlock;
  __shared__ int64_t s_red[BS / 64];
  __shared__ int s_scan[2 * (BS / 64)];
  __shared__ uint32_t s_hist[256];
  __shared__ uint64_t s_keys[kSelectKeyCache];
  __shared__ int s_digit, s_need;

  const int u = blockIdx.x;
  const int tid = threadIdx.x;
  const int r = u / a.Hkv;
  const int g = u - r * a.Hkv;

  int64_t part = 0;
  for (int v = tid; v < u; v += BS) part += unit_info(a, v).count;
  const int64_t offset = block_sum64<BS>(part, s_red);
  const UnitInfo I = unit_info(a, u);
  if (tid == 0) {
    a.sel_indptr[u + 1] = (int32_t)(offset + I.count);
    if (u == 0) a.sel_indptr[0] = 0;
  }
  int32_t* out = a.sel_pages + offset;
  const int n = I.n;

  if (a.mode == kModeAll || a.mode == kModeHeadClass) {
    // ascending union of [0, a_end) and [b_begin, n)
    for (int i = tid; i < I.count; i += BS)
      out[i] = i < I.a_end ? i : I.b_begin + (i - I.a_end);
    return;
  }

  // ranked rules: forced [0, a_end) U [b_begin, n); choose kk of [lo, hi)
  const int lo = I.a_end, hi = I.b_begin;
  const int nn = hi - lo;
  const int forced = lo + (n - hi);
  const int kk = I.count - forced;
  const bool topk = a.mode == kModeTopk;
  const uint64_t sm_seed = splitmix64(a.seed);
  const uint64_t* skeys = a.score_keys + (int64_t)u * a.max_pages;
  auto key_of = [&](int p) -> uint64_t {
    return topk ? skeys[p] : random_key(sm_seed, r, g, p);
  };

  const bool take_all = kk >= nn;
  const bool take_none = kk <= 0;
  const bool cached = nn <= kSelectKeyCache;
  uint64_t T = 0;
  int need = 0;
  if (!take_all && !take_none) {
    if (cached)
      for (int i = tid; i < nn; i += BS) s_keys[i] = key_of(lo + i);
    uint64_t prefix = 0, pmask = 0;
    need = kk;
    for (int shift = 56; shift >= 0; shift -= 8) {
      for (int i = tid; i < 256; i += BS) s_hist[i] = 0u;
      __syncthreads();
      for (int i = tid; i < nn; i += BS) {
        const uint64_t k = cached ? s_keys[i] : key_of(lo + i);
        if ((k & pmask) == prefix) atomicAdd(&s_hist[(k >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (tid < 64) {
        const uint32_t h0 = s_hist[4 * tid], h1 = s_hist[4 * tid + 1];
        const uint32_t h2 = s_hist[4 * tid + 2], h3 = s_hist[4 * tid + 3];
        const int c = (int)(h0 + h1 + h2 + h3);
        int incl = c;
        for (int o = 1; o < 64; o <<= 1) {
          const int y = __shfl_up(incl, o);
          if (tid >= o) incl += y;
        }
        const int excl = incl - c;
        if (excl < need && need <= incl) {
          int rem = need - excl;
          int d = 4 * tid;
          const uint32_t hs[4] = {h0, h1, h2, h3};
          for (int q = 0; q < 4; ++q) {
            if (rem <= (int)hs[q]) { d = 4 * tid + q; break; }
            rem -= (int)hs[q];
          }
          s_digit = d;
          s_need = rem;
        }
      }
      __syncthreads();
      prefix |= (uint64_t)s_digit << shift;
      pmask |= 0xFFull << shift;
      need = s_need;
      __syncthreads();
    }
    T = prefix;
  }

  // ascending emission: forced pages, keys below T, and the first `need` keys equal to T
  int out_base = 0, eq_base = 0;
  for (int c0 = 0; c0 < n; c0 += BS) {
    const int p = c0 + tid;
    const bool in = p < n;
    const bool nonforced = in && p >= lo && p < hi;
    bool lt = false, eq = false;
    if (nonforced && !take_all && !take_none) {
      const uint64_t k = cached ? s_keys[p - lo] : key_of(p);
      lt = k < T;
      eq = k == T;
    }
    int ex_eq, ex_sel, tot_eq, tot_sel;
    // the equal-key rank must be known before the selection flag: two scans
    int dummy_x, dummy_tx;
    block_scan2<BS>(eq, false, ex_eq, dummy_x, tot_eq, dummy_tx, s_scan);
    const bool chosen = take_all || lt || (eq && eq_base + ex_eq < need);
    const bool sel = in && (!nonforced || (!take_none && chosen));
    block_scan2<BS>(sel, false, ex_sel, dummy_x, tot_sel, dummy_tx, s_scan);
    if (sel) out[out_base + ex_sel] = p;
    out_base += tot_sel;
    eq_base += tot_eq;
  }
}

// Mean-key page scores for TOPK_MEANKEY: key of (unit, page p) from
// (q_bar . ksum[phys(p)]) / n_valid(p) in float64, q_bar = sum over the G query
// heads of the request's last query token. Eight lanes per page.
__global__ __launch_bounds__(256) void select_score_kernel(const SelArgs a) {
  __shared__ double s_qbar[128];
  const int u = blockIdx.y;
  const int r = u / a.Hkv;
  const int g = u - r * a.Hkv;
  const int D = a.D;
  const int P = a.P;
  const int max_tokens = a.max_segs * a.pps * P;
  const int L = clampv(a.ctx_lens[r], 0, max_tokens);
  const int n = (L + P - 1) / P;
  const int p_block = blockIdx.x * 256;
  if (p_block >= n) return;
  const int q0 = clampv(a.q_indptr[r], 0, a.total_q);
  const int q1 = clampv(a.q_indptr[r + 1], q0, a.total_q);
  const int tid = threadIdx.x;
  if (tid < D) {
    double s = 0.0;
    if (q1 > q0) {
      const __bf16* qp = a.q + ((int64_t)(q1 - 1) * a.Hq + g * a.G) * D + tid;
      for (int h = 0; h < a.G; ++h) s += (double)(float)qp[(int64_t)h * D];
    }
    s_qbar[tid] = s;
  }
  __syncthreads();
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int sub = lane & 7;           // lane within the page group
  const int per = D / 8;              // floats per lane (16 or 8)
  const int32_t* seg_row = a.seg_table + (int64_t)u * a.max_segs;
  uint64_t* keys = a.score_keys + (int64_t)u * a.max_pages;
  for (int it = 0; it < 8; ++it) {
    const int p = p_block + it * 32 + wave * 8 + (lane >> 3);
    const bool valid = p < n;
    const int ph = valid ? translate_page(seg_row, a.page_table, p, a.pps, a.max_segs, a.n_virtual,
                                          a.n_phys)
                         : -1;
    double dot = 0.0;
    if (ph >= 0) {
      const float* ks = a.page_ksum + (int64_t)ph * D + sub * per;
      for (int i = 0; i < per; i += 4) {
        const float4 v = *reinterpret_cast<const float4*>(ks + i);
        dot = fma((double)v.x, s_qbar[sub * per + i], dot);
        dot = fma((double)v.y, s_qbar[sub * per + i + 1], dot);
        dot = fma((double)v.z, s_qbar[sub * per + i + 2], dot);
        dot = fma((double)v.w, s_qbar[sub * per + i + 3], dot);
      }
    }
    dot += __shfl_xor(dot, 1);
    dot += __shfl_xor(dot, 2);
    dot += __shfl_xor(dot, 4);
    if (valid && sub == 0) {
      const int nvalid = min(P, L - p * P);
      keys[p] = ph >= 0 ? descending_key(dot / (double)nvalid) : ~0ull;
    }
  }
}

hipError_t launch_select_scores(const SelArgs& a, hipStream_t stream) {
  const dim3 grid((a.max_pages + 255) / 256, a.units), block(256);
  hipLaunchKernelGGL(select_score_kernel, grid, block, 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_select_fill(const SelArgs& a, hipStream_t stream) {
  const dim3 grid(a.units), block(kSelectBlock);
  hipLaunchKernelGGL(select_fill_kernel, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace segpa
