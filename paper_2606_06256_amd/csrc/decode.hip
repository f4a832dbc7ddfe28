// Split-KV paged attention for short query chunks (decode), and the
// log-sum-exp combine of split results.
//
// What is computed: Algorithm 2 (SegPagedAttention), FusedVarlenAttention:
// every query row attends to the selected pages of its (request, KV head)
// unit only, in one launch over all units. Section 4.4 gives the exactness of
// merging results over disjoint key subsets with log-sum-exp, which is what
// makes the split over waves exact.
//
// Work decomposition ("stream" split): the selected pages of all units, in
// unit order, form one sequence of 16-token tiles (the CSR sel_indptr times
// tiles per page). Every wave of the grid takes one contiguous, equal share of
// that sequence, so load balance does not depend on how lengths vary between
// units. A wave that covers a whole unit writes the final output; a wave that
// covers part of one writes a normalised partial (o, lse) into slot
// (wave + virtual unit), which is unique because wave ranges are ordered. The
// combine kernel merges the partials of units that span several waves.
//
// The query rows of a unit (row = query * G + head, n_q * G rows) are cut into
// blocks of 16; each (unit, row block) is a virtual unit with the unit's tiles,
// and the tile sequence above runs over virtual units. Decode (n_q * G <= 16)
// has one row block per unit. Per wave and tile one row block forms one
// matrix-core tile:
//   S^T[16 tok x 16 rows] = K_tile[16 x D] . Q^T      (16x16x32 bf16 steps)
//   O^T[D x 16 rows]     += V_tile^T[D x 16] . P^T     (16x16x16 bf16 steps)
// With the K tile stored [D/8][16][8] and the V tile [D][16], each lane's
// operands are contiguous 16-byte / 8-byte loads and the score layout of the
// first product is exactly the operand layout of the second: the softmax needs
// only two cross-lane max steps per tile, and the running max, the sum and the
// rescale are lane-local.
#include "common.hpp"
#include "kernels.hpp"

namespace segpa {

template <int D>
struct KvTile {
  s16x8 k[D / 32];
  s16x4 v[D / 16];
};

// One 16-token tile through buffer descriptors (wave-uniform base in SGPRs).
// Lane (j, grp) takes: K chunk (kb * 4 + grp) of token j (16 B at
// koff + kb * 1024), and V dims nb * 16 + j for tokens 4 * grp .. 4 * grp + 3
// (8 B at voff + nb * 512). range = 0 makes every load return zeros.
template <int D>
__device__ __forceinline__ void load_kv_tile(KvTile<D>& t, const __bf16* kt, const __bf16* vt,
                                             int koff, int voff, int range) {
  const __amdgpu_buffer_rsrc_t kr = make_rsrc(kt, range);
  const __amdgpu_buffer_rsrc_t vr = make_rsrc(vt, range);
#pragma unroll
  for (int kb = 0; kb < D / 32; ++kb)
    t.k[kb] = __builtin_bit_cast(s16x8, __builtin_amdgcn_raw_buffer_load_b128(kr, koff, kb * 1024, 0));
#pragma unroll
  for (int nb = 0; nb < D / 16; ++nb)
    t.v[nb] = __builtin_bit_cast(s16x4, __builtin_amdgcn_raw_buffer_load_b64(vr, voff, nb * 512, 0));
}

// Tiles per wave share: an equal split of all T virtual tiles over the waves,
// but at least kMinChunk tiles so that small problems are not cut into many
// tiny partials (waves past the end get no work).
constexpr int64_t kMinChunk = 8;
__device__ __forceinline__ int64_t stream_chunk(int64_t T, int waves) {
  return max((T + waves - 1) / waves, kMinChunk);
}

// One wave processes unit-local tiles [la, lb) of unit u (nt tiles) for row
// block rb.
template <int D>
__device__ void decode_unit_range(const FwdArgs& a, int u, int rb, int64_t nt, int64_t la,
                                  int64_t lb, int wave, int e_unit0, int e_unit1) {
  constexpr int KB = D / 32;
  constexpr int NB = D / 16;
  const int lane = __lane_id();
  const int j = lane & 15;      // query row of the tile (row = qi * G + h)
  const int grp = lane >> 4;    // lane group: token quad / head-dim chunk
  const int r = u / a.Hkv;
  const int g = u - r * a.Hkv;
  const int G = a.G;
  const int P = a.P;
  const int max_tokens = a.max_segs * a.pps * P;
  const int L = clampv(a.ctx_lens[r], 0, max_tokens);
  const int npg = (L + P - 1) / P;
  const int q0 = clampv(a.q_indptr[r], 0, a.total_q);
  const int nq = clampv(a.q_indptr[r + 1] - q0, 0, min(a.max_q_len, a.total_q - q0));
  const int rows = nq * G;
  const int R = rb * 16 + j;     // row of the unit handled by this lane
  const int qi = R / G;
  const int hh = R - qi * G;
  const bool row_ok = R < rows;
  const int qpos = L - nq + qi;   // last visible position of this row (causal)
  if (rb * 16 >= rows) return;    // row block without rows (shorter chunk)

  // Q operand of the row block (16 rows x D); rows past the chunk read row 0 and are zeroed
  s16x8 qreg[KB];
  {
    const int qrow = row_ok ? qi : 0;
    const int qh = row_ok ? hh : 0;
    const __bf16* qp = a.q + ((int64_t)(q0 + qrow) * a.Hq + g * G + qh) * D + grp * 8;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const s16x8 v = *reinterpret_cast<const s16x8*>(qp + kb * 32);
      const s16x8 z = {0, 0, 0, 0, 0, 0, 0, 0};
      qreg[kb] = row_ok ? v : z;
    }
  }

  const int32_t* seg_row = a.seg_table + (int64_t)u * a.max_segs;
  // The unit's segment-table row, one entry per lane, read alongside the
  // first selected ids: a page's segment lookup is then a lane shuffle, one
  // dependent memory round trip less before the first K/V tile.
  const bool seg_in_regs = a.max_segs <= kWave;
  const int seg_lane = seg_in_regs && lane < a.max_segs ? seg_row[lane] : -1;
  const int koff = (grp * kTile + j) * 16;   // byte offsets inside a tile
  const int voff = j * kTile * 2 + grp * 8;
  const int tpp_log2 = a.tpp_log2;
  const int tpp_mask = (1 << tpp_log2) - 1;

  float m = -INFINITY;
  float lsum = 0.f;
  f32x4 acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = (f32x4){0.f, 0.f, 0.f, 0.f};

  // one tile step: scores, online softmax update, P.V accumulation
  auto step = [&](const KvTile<D>& tile, int jpg, int ph, int sub) {
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) s = mfma16x16x32(tile.k[kb], qreg[kb], s);
    // this lane holds row j, tokens 4*grp + 0..3 of the tile
    const int lim = ph >= 0 ? min(L - 1, qpos) : -1;   // last visible position
    const int tok0 = jpg * P + sub * kTile + grp * 4;
    float sv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) sv[e] = tok0 + e <= lim ? s[e] * a.scale_log2 : -INFINITY;
    float mx = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = fast_exp2(m - m_use);
    const float p0 = fast_exp2(sv[0] - m_use);
    const float p1 = fast_exp2(sv[1] - m_use);
    const float p2 = fast_exp2(sv[2] - m_use);
    const float p3 = fast_exp2(sv[3] - m_use);
    lsum = lsum * alpha + ((p0 + p1) + (p2 + p3));
    m = m_new;
    const s16x4 pb = pack_bf16x4(p0, p1, p2, p3);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      acc[nb] *= alpha;
      acc[nb] = mfma16x16x16(tile.v[nb], pb, acc[nb]);
    }
  };

  // Pages are translated 64 at a time (one per lane: selected id ->
  // segment -> virtual -> physical); tiles then stream through two register
  // buffers, loading tile t+1 while tile t is computed.
  const int64_t e_first = la >> tpp_log2;
  const int64_t e_last = (lb - 1) >> tpp_log2;
  for (int64_t eb = e_first; eb <= e_last; eb += kWave) {
    int b_jpg = eb + lane <= e_last ? a.sel_pages[e_unit0 + eb + lane] : -1;
    if (!(b_jpg >= 0 && b_jpg < npg)) b_jpg = -1;
    int b_ph = -1;
    if (seg_in_regs) {
      // (the shuffle runs with every lane active; jp < npg keeps s < max_segs)
      const int sidx = b_jpg >= 0 ? b_jpg / a.pps : 0;
      const int v0 = __shfl(seg_lane, sidx);
      if (b_jpg >= 0 && v0 >= 0) {
        const int64_t vp = (int64_t)v0 + (b_jpg - sidx * a.pps);
        if (vp < a.n_virtual) {
          const int ph = a.page_table[vp];
          b_ph = ph >= 0 && (int64_t)ph < a.n_phys ? ph : -1;
        }
      }
    } else if (b_jpg >= 0) {
      b_ph = translate_page(seg_row, a.page_table, b_jpg, a.pps, a.max_segs, a.n_virtual, a.n_phys);
    }
    const int64_t t0 = max(la, eb << tpp_log2);
    const int64_t t1 = min(lb, (eb + kWave) << tpp_log2);
    auto fetch = [&](KvTile<D>& tile, int64_t t, int& jpg, int& ph, int& sub) {
      const int idx = (int)((t >> tpp_log2) - eb);
      jpg = __builtin_amdgcn_readlane(b_jpg, idx);
      ph = __builtin_amdgcn_readlane(b_ph, idx);
      sub = (int)(t & tpp_mask);
      // an unusable page reads as zeros; so do V slots past the context (their
      // probability is 0, and stale contents there must not reach the sum)
      const int64_t base = uniform64(((int64_t)(ph < 0 ? 0 : ph) * P + sub * kTile) * D);
      load_kv_tile<D>(tile, a.k_pool + base, a.v_pool + base, koff, voff,
                      ph >= 0 ? kTile * D * 2 : 0);
      const int valid = L - (jpg * P + sub * kTile);   // tokens of the tile inside the context
      if (ph >= 0 && valid < kTile) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (grp * 4 + e >= valid) tile.v[nb][e] = 0;
      }
    };
    // Loads are issued unconditionally (past the end they re-read the last
    // tile, already in cache) so that every compute step waits only for its
    // own buffer while the other buffer's loads stay in flight.
    KvTile<D> ta_buf, tb_buf;
    int x_jpg, x_ph, x_sub, y_jpg, y_ph, y_sub;
    // The scheduling barriers keep each buffer's loads ahead of the other
    // buffer's compute (the scheduler would otherwise sink them to their use).
    fetch(ta_buf, t0, x_jpg, x_ph, x_sub);
    for (int64_t t = t0; t < t1; t += 2) {
      fetch(tb_buf, min(t + 1, t1 - 1), y_jpg, y_ph, y_sub);
      __builtin_amdgcn_sched_barrier(0);
      step(ta_buf, x_jpg, x_ph, x_sub);
      __builtin_amdgcn_sched_barrier(0);
      fetch(ta_buf, min(t + 2, t1 - 1), x_jpg, x_ph, x_sub);
      __builtin_amdgcn_sched_barrier(0);
      if (t + 1 < t1) step(tb_buf, y_jpg, y_ph, y_sub);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // row totals: the four lane groups hold disjoint token subsets
  float ltot = lsum + __shfl_xor(lsum, 16);
  ltot += __shfl_xor(ltot, 32);
  const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
  const float lse2 = ltot > 0.f ? m + __log2f(ltot) : -INFINITY;
  if (!row_ok) return;
  if (la == 0 && lb == nt) {
    __bf16* op = a.out + ((int64_t)(q0 + qi) * a.Hq + g * G + hh) * D;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const s16x4 o = pack_bf16x4(acc[nb][0] * inv, acc[nb][1] * inv, acc[nb][2] * inv,
                                  acc[nb][3] * inv);
      *reinterpret_cast<s16x4*>(op + nb * 16 + grp * 4) = o;
    }
    if (grp == 0 && a.lse != nullptr) a.lse[(int64_t)(q0 + qi) * a.Hq + g * G + hh] = lse2 * kLn2;
  } else {
    const int64_t slot = (int64_t)wave + (int64_t)u * a.row_blocks + rb;
    float* po = a.part_o + (slot * 16 + j) * D;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const f32x4 o = acc[nb] * inv;
      *reinterpret_cast<f32x4*>(po + nb * 16 + grp * 4) = o;
    }
    if (grp == 0) a.part_lse[slot * 16 + j] = lse2;
  }
}

template <int D>
__global__ __launch_bounds__(kDecodeBlock) void decode_attn_kernel(const FwdArgs a) {
  extern __shared__ int32_t s_indptr[];
  const int U = a.units;
  for (int i = threadIdx.x; i <= U; i += blockDim.x)
    s_indptr[i] = (int32_t)clampv<int64_t>(a.sel_indptr[i], 0, a.sel_capacity);
  __syncthreads();

  const int RB = a.row_blocks;
  const int wave = blockIdx.x * (kDecodeBlock / kWave) + (threadIdx.x >> 6);
  const int64_t T = ((int64_t)s_indptr[U] << a.tpp_log2) * RB;   // virtual tiles
  const int64_t chunk = stream_chunk(T, a.total_waves);
  const int64_t t_begin = (int64_t)wave * chunk;
  const int64_t t_end = min(T, t_begin + chunk);
  if (t_begin >= t_end) return;

  // last unit whose first entry is <= the entry of the wave's first tile
  const int64_t e_begin = (t_begin / RB) >> a.tpp_log2;
  int lo = 0, hi = U - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_indptr[mid] <= e_begin) lo = mid; else hi = mid - 1;
  }
  for (int u = lo; u < U; ++u) {
    const int e0 = s_indptr[u];
    const int e1 = s_indptr[u + 1];
    const int64_t ut0 = ((int64_t)e0 << a.tpp_log2) * RB;   // virtual range of unit u
    const int64_t nt = ((int64_t)(e1 - e0)) << a.tpp_log2;   // tiles per row block
    if (ut0 >= t_end) break;
    if (nt <= 0) continue;
    const int64_t ut1 = ut0 + nt * RB;
    if (ut1 <= t_begin) continue;
    const int rb0 = (int)((max(t_begin, ut0) - ut0) / nt);
    for (int rb = rb0; rb < RB; ++rb) {
      const int64_t vt0 = ut0 + (int64_t)rb * nt;
      if (vt0 >= t_end) break;
      const int64_t ta = max(t_begin, vt0);
      const int64_t tb = min(t_end, vt0 + nt);
      if (ta >= tb) continue;
      decode_unit_range<D>(a, u, rb, nt, ta - vt0, tb - vt0, wave, e0, e1);
    }
  }
}

// Merge the split partials of every virtual unit (unit, row block) that spans
// several waves (log-sum-exp, Section 4.4); write O = 0, LSE = -inf for units
// without selected tiles. One block per virtual unit, 16 threads per query row,
// each with D / 16 output dims. A thread issues the row LSEs and its dims of 8
// partials at once (no load waits for another), so a batch of 8 partials
// costs one memory round trip; batches are merged in wave order with one
// rescale each, so the result does not depend on timing.
template <int D>
__global__ __launch_bounds__(256) void combine_kernel(const FwdArgs a) {
  constexpr int kRows = 16;
  constexpr int TPR = 256 / kRows;     // threads per row
  constexpr int NQ = D / TPR / 4;      // float4 groups per thread
  constexpr int WB = 8;                // partials per batch
  const int RB = a.row_blocks;
  const int v = blockIdx.x;
  const int u = v / RB;
  const int rb = v - u * RB;
  const int U = a.units;
  const int64_t cap = a.sel_capacity;
  const int64_t e_tot = clampv<int64_t>(a.sel_indptr[U], 0, cap);
  const int64_t e0 = clampv<int64_t>(a.sel_indptr[u], 0, cap);
  const int64_t e1 = clampv<int64_t>(a.sel_indptr[u + 1], 0, cap);
  const int64_t T = (e_tot << a.tpp_log2) * RB;
  const int64_t nt = (e1 - e0) << a.tpp_log2;
  const int64_t vt0 = (e0 << a.tpp_log2) * RB + (int64_t)rb * nt;
  const int r = u / a.Hkv;
  const int g = u - r * a.Hkv;
  const int G = a.G;
  const int q0 = clampv(a.q_indptr[r], 0, a.total_q);
  const int nq = clampv(a.q_indptr[r + 1] - q0, 0, min(a.max_q_len, a.total_q - q0));
  const int row = threadIdx.x / TPR;
  const int d0 = (threadIdx.x % TPR) * (4 * NQ);
  const int R = rb * kRows + row;
  if (R >= nq * G) return;

  // must mirror the decode kernel's partition
  const bool empty = nt <= 0;
  int64_t w0 = 0, nw = 0;
  if (!empty) {
    const int64_t chunk = stream_chunk(T, a.total_waves);
    w0 = vt0 / chunk;
    nw = (vt0 + nt - 1) / chunk - w0 + 1;
    if (nw == 1) return;   // one wave wrote the final output
  }
  const int64_t sbase = (int64_t)u * RB + rb + w0;   // slot of the first partial
  float M = -INFINITY, Z = 0.f;
  f32x4 o[NQ];
#pragma unroll
  for (int i = 0; i < NQ; ++i) o[i] = (f32x4){0.f, 0.f, 0.f, 0.f};
  for (int64_t w = 0; w < nw; w += WB) {
    float x[WB];
    f32x4 po[WB][NQ];
#pragma unroll
    for (int k = 0; k < WB; ++k) {
      const int64_t s = sbase + min(w + k, nw - 1);
      x[k] = w + k < nw ? a.part_lse[s * kRows + row] : -INFINITY;
#pragma unroll
      for (int i = 0; i < NQ; ++i)
        po[k][i] = *reinterpret_cast<const f32x4*>(a.part_o + (s * kRows + row) * D + d0 + 4 * i);
    }
    float mb = M;
#pragma unroll
    for (int k = 0; k < WB; ++k) mb = fmaxf(mb, x[k]);
    if (mb == -INFINITY) continue;             // nothing visible so far
    const float sc = fast_exp2(M - mb);        // 0 while M is -inf
    Z *= sc;
#pragma unroll
    for (int i = 0; i < NQ; ++i) o[i] *= sc;
#pragma unroll
    for (int k = 0; k < WB; ++k) {
      const float wt = fast_exp2(x[k] - mb);  // 0 for x = -inf
      Z += wt;
#pragma unroll
      for (int i = 0; i < NQ; ++i) o[i] += wt * po[k][i];
    }
    M = mb;
  }
  const int qi = R / G;
  const int hh = R - qi * G;
  const int64_t orow = (int64_t)(q0 + qi) * a.Hq + g * G + hh;
  const float iz = Z > 0.f ? 1.f / Z : 0.f;
#pragma unroll
  for (int i = 0; i < NQ; ++i)
    *reinterpret_cast<s16x4*>(a.out + orow * D + d0 + 4 * i) =
        pack_bf16x4(o[i][0] * iz, o[i][1] * iz, o[i][2] * iz, o[i][3] * iz);
  if (d0 == 0 && a.lse != nullptr) a.lse[orow] = Z > 0.f ? (M + __log2f(Z)) * kLn2 : -INFINITY;
}

hipError_t launch_decode(const FwdArgs& a, hipStream_t stream) {
  const size_t lds = (size_t)(a.units + 1) * sizeof(int32_t);
  const dim3 grid(a.total_waves / (kDecodeBlock / kWave)), block(kDecodeBlock);
  if (a.D == 128)
    launch(decode_attn_kernel<128>, grid, block, lds, stream, a);
  else
    launch(decode_attn_kernel<64>, grid, block, lds, stream, a);
  return hipGetLastError();
}

hipError_t launch_combine(const FwdArgs& a, hipStream_t stream) {
  const dim3 grid(a.units * a.row_blocks), block(256);
  if (a.D == 128)
    launch(combine_kernel<128>, grid, block, 0, stream, a);
  else
    launch(combine_kernel<64>, grid, block, 0, stream, a);
  return hipGetLastError();
}

int decode_blocks_per_cu(int D, int units) {
  const size_t lds = (size_t)(units + 1) * sizeof(int32_t);
  int n = 0;
  hipError_t e;
  if (D == 128)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, decode_attn_kernel<128>, kDecodeBlock, lds);
  else
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, decode_attn_kernel<64>, kDecodeBlock, lds);
  if (e != hipSuccess || n < 1) return 1;
  return n;
}

}  // namespace segpa
