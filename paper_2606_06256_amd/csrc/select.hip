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
// (key, page) pair by a radix select (LDS histograms; a 12-bit first digit,
// then 8-bit digits over a shrinking candidate list, then an exact rank among
// at most 128 candidates) and then emit the chosen pages in ascending order
// with block-wide prefix counts.
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

// The per-unit inputs of the closed-form counts, read in one go so that a
// block can issue them early and do the arithmetic later.
struct UnitRaw {
  int L;        // context length (unclamped)
  int q0, q1;   // HEAD_CLASS: query range of the request
  int local;    // HEAD_CLASS: 1 for a local head
  int budget;   // RANDOM_HASH / TOPK: budget of the request
};

__device__ UnitRaw load_unit(const SelArgs& a, int u) {
  const int r = u / a.Hkv;
  const int g = u - r * a.Hkv;
  UnitRaw x{a.ctx_lens[r], 0, 1, 0, 0};
  if (a.mode == kModeHeadClass) {
    x.local = a.head_policy[g] == 0;
    if (a.q_indptr != nullptr) { x.q0 = a.q_indptr[r]; x.q1 = a.q_indptr[r + 1]; }
  } else if (a.mode == kModeRandom || a.mode == kModeTopk) {
    x.budget = a.budget[r];
  }
  return x;
}

__device__ UnitInfo unit_info_of(const SelArgs& a, const UnitRaw& x) {
  const int max_tokens = a.max_segs * a.pps * a.P;
  const int L = clampv(x.L, 0, max_tokens);
  UnitInfo I;
  I.n = (L + a.P - 1) / a.P;
  I.count = I.n;
  I.a_end = I.n;
  I.b_begin = I.n;
  if (a.mode == kModeHeadClass) {
    if (x.local) {
      const int nq = clampv(x.q1 - x.q0, 0, L);
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
    const int b = max(0, x.budget);
    I.a_end = fh;
    I.b_begin = max(fh, I.n - ft);
    I.count = min(I.n, max(b, forced));
  }
  return I;
}

__device__ UnitInfo unit_info(const SelArgs& a, int u) { return unit_info_of(a, load_unit(a, u)); }

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

}  // namespace

__global__ __launch_bounds__(kSelectBlock) void select_fill_kernel(const SelArgs a) {
  constexpr int BS = kSelectBlock;
  __shared__ int64_t s_red[BS / 64];
  __shared__ int s_scan[BS / 64];
  __shared__ uint32_t s_hist[4096];
  // key cache of the candidates [lo, hi): whole keys for up to
  // kSelectKeyCache / 2 of them, else the high halves of up to kSelectKeyCache
  __shared__ uint64_t s_kc[kSelectKeyCache / 2];
  __shared__ uint64_t s_ck[kSelectCand], s_ck2[kSelectCand];
  __shared__ int s_ci[kSelectCand], s_ci2[kSelectCand];
  __shared__ int s_digit, s_need, s_count, s_fill, s_tidx;
  __shared__ uint64_t s_tkey;

  const int u = blockIdx.x;
  const int tid = threadIdx.x;
  const int r = u / a.Hkv;
  const int g = u - r * a.Hkv;

  // CSR offset = the counts of the earlier units. The inputs of the first
  // kPre of them per thread are loaded here and summed only before the
  // output is written, so their latency overlaps the ranking.
  constexpr int kPre = 2;
  UnitRaw pre[kPre];
#pragma unroll
  for (int k = 0; k < kPre; ++k) {
    const int v = tid + k * BS;
    if (v < u) pre[k] = load_unit(a, v);
  }
  auto csr_offset = [&]() -> int64_t {
    int64_t part = 0;
#pragma unroll
    for (int k = 0; k < kPre; ++k)
      if (tid + k * BS < u) part += unit_info_of(a, pre[k]).count;
    for (int v = tid + kPre * BS; v < u; v += BS) part += unit_info(a, v).count;
    return block_sum64<BS>(part, s_red);
  };
  const UnitInfo I = unit_info(a, u);
  const int n = I.n;

  if (a.mode == kModeAll || a.mode == kModeHeadClass) {
    const int64_t offset = csr_offset();
    if (tid == 0) {
      a.sel_indptr[u + 1] = (int32_t)(offset + I.count);
      if (u == 0) a.sel_indptr[0] = 0;
    }
    int32_t* out = a.sel_pages + offset;
    // ascending union of [0, a_end) and [b_begin, n)
    for (int i = tid; i < I.count; i += BS)
      out[i] = i < I.a_end ? i : I.b_begin + (i - I.a_end);
    return;
  }

  // ranked rules: forced [0, a_end) U [b_begin, n); choose kk of [lo, hi).
  // The choice is the kk smallest (key, page) pairs: find the kk-th smallest
  // pair (T, pT) exactly, then keep every pair <= (T, pT).
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
  // Units of up to kSelectKeyCache / 2 candidates keep whole keys in LDS.
  // Larger ones, up to kSelectKeyCache, keep the high 32 bits of each key:
  // they decide every radix pass whose digits lie in the high half, and the
  // emission except for keys whose high half equals the threshold's; whole
  // keys are recomputed (or re-read) only for the candidates left in the
  // threshold's bin and for such ties. Longer units recompute every key.
  const bool whole = nn <= kSelectKeyCache / 2;
  const bool cached = nn <= kSelectKeyCache;
  constexpr int kU = 4;   // keys per thread handled together in the full passes
  uint32_t* s_khi = reinterpret_cast<uint32_t*>(s_kc);
  uint64_t T = 0;
  int pT = -1;
  if (!take_all && !take_none) {
    // cached keys: the histogram of the first (12-bit) digit is built while
    // the keys are computed
    if (cached) {
      for (int i = tid; i < 4096; i += BS) s_hist[i] = 0u;
      if (tid == 0) s_fill = 0;
      __syncthreads();
      // kU keys per thread at a time: their hashes (or loads) are independent
      for (int i0 = tid; i0 < nn; i0 += kU * BS) {
        uint64_t kv[kU];
#pragma unroll
        for (int e = 0; e < kU; ++e) kv[e] = i0 + e * BS < nn ? key_of(lo + i0 + e * BS) : 0;
#pragma unroll
        for (int e = 0; e < kU; ++e) {
          const int i = i0 + e * BS;
          if (i < nn) {
            if (whole) s_kc[i] = kv[e]; else s_khi[i] = (uint32_t)(kv[e] >> 32);
            atomicAdd(&s_hist[(uint32_t)(kv[e] >> 52)], 1u);
          }
        }
      }
    }
    __syncthreads();
    auto key_full = [&](int i) -> uint64_t { return whole ? s_kc[i] : key_of(lo + i); };
    // a key for a pass whose fixed bits and digit all lie at bit 32 or above:
    // its high half suffices (the low half may read as zero)
    auto key_high = [&](int i) -> uint64_t {
      return whole ? s_kc[i] : cached ? (uint64_t)s_khi[i] << 32 : key_of(lo + i);
    };
    // Radix passes narrow the candidates (keys that match `prefix` on the bits
    // of `pmask`): the first pass over all keys with a 12-bit digit, the next
    // ones with 8-bit digits, until at most kRankMax candidates remain or the
    // whole key is fixed. Candidates go to an LDS list once they fit in it.
    constexpr int kRankMax = 128;
    uint64_t prefix = 0, pmask = 0;
    int need = kk;                  // rank (1-based) of the threshold among candidates
    int shift = 64;
    int ncand = nn;
    bool listed = false;            // candidates in s_ck/s_ci, else: filter [lo, hi)
    while (ncand > kRankMax && shift > 0) {
      // a 12-bit first digit, then 8-bit digits; the last one takes the 4
      // bits that remain (52 = 6 x 8 + 4), so the shift never goes below 0
      const int bits = (shift == 64) ? 12 : min(8, shift);
      const int nb = 1 << bits;
      const bool prebuilt = cached && shift == 64;
      shift -= bits;
      const int len = listed ? ncand : nn;
      // every bit this pass reads (the fixed prefix and the digit) is at shift or above
      const bool high = shift >= 32;
      auto key_pass = [&](int i) -> uint64_t { return high ? key_high(i) : key_full(i); };
      if (!prebuilt) {
        for (int i = tid; i < nb; i += BS) s_hist[i] = 0u;
        if (tid == 0) s_fill = 0;
        __syncthreads();
        if (listed) {
          for (int i = tid; i < len; i += BS)
            atomicAdd(&s_hist[(uint32_t)(s_ck[i] >> shift) & (uint32_t)(nb - 1)], 1u);
        } else {
          for (int i0 = tid; i0 < len; i0 += kU * BS) {
            uint64_t kv[kU];
#pragma unroll
            for (int e = 0; e < kU; ++e) kv[e] = i0 + e * BS < len ? key_pass(i0 + e * BS) : 0;
#pragma unroll
            for (int e = 0; e < kU; ++e)
              if (i0 + e * BS < len && (kv[e] & pmask) == prefix)
                atomicAdd(&s_hist[(uint32_t)(kv[e] >> shift) & (uint32_t)(nb - 1)], 1u);
          }
        }
        __syncthreads();
      }
      // the bin that holds the need-th candidate: block-wide scan of bin groups
      {
        const int per = nb >= BS ? nb / BS : 1;
        int c = 0;
        if (tid * per < nb)
          for (int q = 0; q < per; ++q) c += (int)s_hist[tid * per + q];
        int ex, tot;
        block_scan<BS>(c, ex, tot, s_scan);
        if (c > 0 && ex < need && need <= ex + c) {
          int rem = need - ex, d = tid * per;
          for (int q = 0; q < per; ++q) {
            const int h = (int)s_hist[tid * per + q];
            if (rem <= h) { d = tid * per + q; break; }
            rem -= h;
          }
          s_digit = d;
          s_need = rem;
          s_count = (int)s_hist[d];
        }
      }
      __syncthreads();
      need = s_need;
      const int newc = s_count;
      prefix |= (uint64_t)s_digit << shift;
      pmask |= (uint64_t)(nb - 1) << shift;
      if (newc <= kSelectCand) {
        // unordered compaction of the survivors (order is irrelevant here);
        // straight into the list unless the list itself is being read
        if (listed) {
          for (int i = tid; i < len; i += BS) {
            const uint64_t k = s_ck[i];
            if ((k & pmask) == prefix) {
              const int slot = atomicAdd(&s_fill, 1);
              s_ck2[slot] = k;
              s_ci2[slot] = s_ci[i];
            }
          }
        } else {
          for (int i0 = tid; i0 < len; i0 += kU * BS) {
            uint64_t kv[kU];
#pragma unroll
            for (int e = 0; e < kU; ++e) kv[e] = i0 + e * BS < len ? key_pass(i0 + e * BS) : 0;
#pragma unroll
            for (int e = 0; e < kU; ++e) {
              const int i = i0 + e * BS;
              if (i < len && (kv[e] & pmask) == prefix) {
                const int slot = atomicAdd(&s_fill, 1);
                s_ck[slot] = key_full(i);          // the list holds full keys
                s_ci[slot] = lo + i;
              }
            }
          }
        }
        __syncthreads();
        if (listed) {
          for (int i = tid; i < newc; i += BS) { s_ck[i] = s_ck2[i]; s_ci[i] = s_ci2[i]; }
          __syncthreads();
        }
        listed = true;
      }
      ncand = newc;
    }
    if (shift == 0) {
      // every candidate holds the key `prefix`: the threshold is the need-th
      // lowest page index among them
      if (tid == 0) { s_tkey = prefix; s_tidx = -1; }
      int base = 0;
      for (int c0 = 0; c0 < nn; c0 += BS) {
        const int i = c0 + tid;
        const bool m = i < nn && key_full(i) == prefix;
        int ex, tot;
        block_scan<BS>(m ? 1 : 0, ex, tot, s_scan);
        if (m && base + ex == need - 1) s_tidx = lo + i;
        base += tot;
        if (base >= need) break;
      }
    } else {
      if (!listed) {
        // the loop did not run: nn <= kRankMax, every key is a candidate
        for (int i = tid; i < nn; i += BS) { s_ck[i] = key_full(i); s_ci[i] = lo + i; }
        __syncthreads();
      }
      // exact rank of each candidate pair (key, page) among the candidates
      if (tid < ncand) {
        const uint64_t k = s_ck[tid];
        const int idx = s_ci[tid];
        int rank = 0;
        for (int i = 0; i < ncand; ++i) {
          const uint64_t ko = s_ck[i];
          rank += (ko < k || (ko == k && s_ci[i] < idx)) ? 1 : 0;
        }
        if (rank == need - 1) { s_tkey = k; s_tidx = idx; }
      }
    }
    __syncthreads();
    T = s_tkey;
    pT = s_tidx;
  }

  const int64_t offset = csr_offset();
  if (tid == 0) {
    a.sel_indptr[u + 1] = (int32_t)(offset + I.count);
    if (u == 0) a.sel_indptr[0] = 0;
  }
  int32_t* out = a.sel_pages + offset;

  // ascending emission: forced pages and the chosen pages, four consecutive
  // pages per thread (one block prefix count per 4 * BS pages)
  constexpr int kPer = 4;
  int out_base = 0;
  for (int c0 = 0; c0 < n; c0 += kPer * BS) {
    bool sel[kPer];
    int cnt = 0;
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
      const int p = c0 + tid * kPer + e;
      const bool in = p < n;
      const bool nonforced = in && p >= lo && p < hi;
      sel[e] = in && !nonforced;
      if (nonforced) {
        if (take_all) sel[e] = true;
        else if (!take_none) {
          if (whole) {
            const uint64_t k = s_kc[p - lo];
            sel[e] = k < T || (k == T && p <= pT);
          } else {
            const uint32_t khi = cached ? s_khi[p - lo] : (uint32_t)(key_of(p) >> 32);
            const uint32_t thi = (uint32_t)(T >> 32);
            if (khi != thi) {
              sel[e] = khi < thi;
            } else {
              const uint64_t k = key_of(p);
              sel[e] = k < T || (k == T && p <= pT);
            }
          }
        }
      }
      cnt += sel[e] ? 1 : 0;
    }
    int ex, tot;
    block_scan<BS>(cnt, ex, tot, s_scan);
    int o = out_base + ex;
#pragma unroll
    for (int e = 0; e < kPer; ++e)
      if (sel[e]) out[o++] = c0 + tid * kPer + e;
    out_base += tot;
  }
}

// Mean-key page scores for TOPK_MEANKEY: key of (unit, page p) from
// (q_bar . ksum[phys(p)]) / n_valid(p) in float64, q_bar = sum over the G query
// heads of the request's last query token. Eight lanes per page.
__global__ __launch_bounds__(256) void select_score_kernel(const SelArgs a) {
  constexpr int BS = 256;
  constexpr int kRows = 8;            // pages per lane group loaded before any arithmetic
  __shared__ double s_qbar[128];
  __shared__ int s_ph[BS];
  const int u = blockIdx.y;
  const int r = u / a.Hkv;
  const int g = u - r * a.Hkv;
  const int D = a.D;
  const int P = a.P;
  const int max_tokens = a.max_segs * a.pps * P;
  const int L = clampv(a.ctx_lens[r], 0, max_tokens);
  const int n = (L + P - 1) / P;
  const int p_block = blockIdx.x * BS;
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
  // every page of the block translated at once (one per thread), so the
  // key-sum loads below do not wait on a table lookup each
  {
    const int p = p_block + tid;
    const int32_t* seg_row = a.seg_table + (int64_t)u * a.max_segs;
    s_ph[tid] = p < n ? translate_page(seg_row, a.page_table, p, a.pps, a.max_segs, a.n_virtual, a.n_phys)
                      : -1;
  }
  __syncthreads();
  // 16 lanes per page, D / 16 consecutive floats each (two or one 16-byte loads)
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int grp = lane >> 4;          // page within a row of 4
  const int sub = lane & 15;
  const int per = D / 16;
  double qb[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) qb[i] = i < per ? s_qbar[sub * per + i] : 0.0;
  uint64_t* keys = a.score_keys + (int64_t)u * a.max_pages;
  // wave w covers block pages [64 w, 64 w + 64): rows of 4 pages
  for (int r0 = 0; r0 < 16; r0 += kRows) {
    float4 v[kRows][2];
#pragma unroll
    for (int k = 0; k < kRows; ++k) {
      const int ph = s_ph[wave * 64 + (r0 + k) * 4 + grp];
      const float4 z = {0.f, 0.f, 0.f, 0.f};
      v[k][0] = z;
      v[k][1] = z;
      if (ph >= 0) {
        const float* ks = a.page_ksum + (int64_t)ph * D + sub * per;
        v[k][0] = *reinterpret_cast<const float4*>(ks);
        if (per == 8) v[k][1] = *reinterpret_cast<const float4*>(ks + 4);
      }
    }
#pragma unroll
    for (int k = 0; k < kRows; ++k) {
      double dot = 0.0;
      dot = fma((double)v[k][0].x, qb[0], dot);
      dot = fma((double)v[k][0].y, qb[1], dot);
      dot = fma((double)v[k][0].z, qb[2], dot);
      dot = fma((double)v[k][0].w, qb[3], dot);
      dot = fma((double)v[k][1].x, qb[4], dot);
      dot = fma((double)v[k][1].y, qb[5], dot);
      dot = fma((double)v[k][1].z, qb[6], dot);
      dot = fma((double)v[k][1].w, qb[7], dot);
      dot += __shfl_xor(dot, 1);
      dot += __shfl_xor(dot, 2);
      dot += __shfl_xor(dot, 4);
      dot += __shfl_xor(dot, 8);
      const int pi = wave * 64 + (r0 + k) * 4 + grp;
      const int p = p_block + pi;
      if (sub == 0 && p < n) {
        const int ph = s_ph[pi];
        const int nvalid = min(P, L - p * P);
        keys[p] = ph >= 0 ? descending_key(dot / (double)nvalid) : ~0ull;
      }
    }
  }
}

hipError_t launch_select_scores(const SelArgs& a, hipStream_t stream) {
  const dim3 grid((a.max_pages + 255) / 256, a.units), block(256);
  launch(select_score_kernel, grid, block, 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_select_fill(const SelArgs& a, hipStream_t stream) {
  const dim3 grid(a.units), block(kSelectBlock);
  launch(select_fill_kernel, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace segpa
