// Chunked prefill over a sparse, paged context: many query rows per unit.
//
// What is computed: the same attention as the decode kernel (Algorithm 2,
// FusedVarlenAttention over each head's own selected pages; causal inside the
// query chunk, which sits at the end of the context). Prefill is where the
// paper reports its largest gains, because the quadratic work follows the
// attended keys (Section 5.3). Here the work is a dense contraction, so it
// runs on the matrix cores.
//
// One block per (unit, 256 query rows); 8 waves, 32 rows each (row = query *
// G + head, so a GQA group shares its KV head). The unit's selected pages are
// translated once per chunk of entries into LDS. Keys stream in steps of 32
// (two 16-token tiles): the block copies the step's K and V tiles into one of
// two LDS stages while the waves compute on the other. Per wave and step:
//   S^T[32 keys x 32 rows]  = K_step[32 x D] . Q^T       (D/16 steps, 32x32x16)
//   O^T[D x 32 rows]       += V_step^T[D x 32] . P^T     (2 x D/32, 32x32x16)
// In the S^T layout each lane holds 16 keys of one row, so the row max needs
// one cross-half swap and the running max, the sum and the rescale are
// lane-local; the 16 probabilities are, in order, the operand of the second
// product (the key order inside a step is permuted identically for V).
#include "common.hpp"
#include "kernels.hpp"

namespace segpa {

typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f32x16 mfma32x32x16(s16x8 a, s16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// value of lane l ^ 32 (v_permlane32_swap)
__device__ __forceinline__ float swap_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(__lane_id() < 32 ? r[1] : r[0]);
}

constexpr int kPfWaves = 8;
constexpr int kPfThreads = kPfWaves * 64;
constexpr int kPfRows = kPfWaves * 32;     // query rows per block
constexpr int kPfEntries = 1024;           // translated page entries held in LDS

template <int D>
__global__ __launch_bounds__(kPfThreads, 1) void prefill_kernel(const FwdArgs a) {
  constexpr int KS = D / 16;               // QK steps (16 dims each)
  constexpr int NDB = D / 32;              // 32-dim blocks of the output
  constexpr int TB = kTile * D * 2;        // bytes per tile
  __shared__ __attribute__((aligned(16))) char s_kv[2][4 * TB];   // stage: K0 K1 V0 V1
  __shared__ int s_pos[kPfEntries];        // first token position of each entry's page, -1 unusable
  __shared__ int s_phys[kPfEntries];

  // (unit, row block); blocks of one unit are dealt to the same XCD so that
  // its KV stays in that XCD's L2 while they stream it together
  const int RBP = a.row_blocks;
  const int nblk = gridDim.x;
  const int b = blockIdx.x;
  const int v = (nblk % 8 == 0) ? (b % 8) * (nblk / 8) + b / 8 : b;
  const int u = v / RBP;
  const int rb = v - u * RBP;
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
  const int R0 = rb * kPfRows;
  if (R0 >= rows) return;                  // block-uniform

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int j = lane & 31;                 // row within the wave
  const int hf = lane >> 5;                // lane half
  const int R = R0 + w * 32 + j;
  const bool row_ok = R < rows;
  const int qi = (row_ok ? R : R0) / G;
  const int hh = (row_ok ? R : R0) - qi * G;
  const int vis_row = min(L - 1, L - nq + qi);          // last visible position of this row
  const int vis_lo = min(L - 1, L - nq + R0 / G);       // smallest over the block
  const int vis_hi = min(L - 1, L - nq + (min(rows, R0 + kPfRows) - 1) / G);

  // Q^T operand: lane holds Q[row j][16 s + 8 hf .. + 8]
  s16x8 qreg[KS];
  {
    const __bf16* qp = a.q + ((int64_t)(q0 + qi) * a.Hq + g * G + hh) * D + hf * 8;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const s16x8 x = *reinterpret_cast<const s16x8*>(qp + s * 16);
      const s16x8 z = {0, 0, 0, 0, 0, 0, 0, 0};
      qreg[s] = row_ok ? x : z;
    }
  }

  const int U = a.units;
  const int64_t cap = a.sel_capacity;
  const int e0 = (int)clampv<int64_t>(a.sel_indptr[u], 0, cap);
  const int e1 = (int)clampv<int64_t>(a.sel_indptr[u + 1], 0, cap);
  const int n_e = max(0, e1 - e0);
  const int32_t* seg_row = a.seg_table + (int64_t)u * a.max_segs;
  const int tpp_log2 = a.tpp_log2;
  const int tpp = 1 << tpp_log2;
  const float c = a.scale_log2;
  (void)U;

  float m = -INFINITY;                     // running max of raw scores of row j
  float lsum = 0.f;
  f32x16 acc[NDB];
#pragma unroll
  for (int d = 0; d < NDB; ++d) acc[d] = (f32x16){};

  bool done = false;
  for (int ce = 0; ce < n_e && !done; ce += kPfEntries) {
    const int cn = min(kPfEntries, n_e - ce);
    __syncthreads();                       // previous chunk no longer read
    for (int i = tid; i < cn; i += kPfThreads) {
      const int jp = a.sel_pages[e0 + ce + i];
      int ph = -1;
      if (jp >= 0 && jp < npg)
        ph = translate_page(seg_row, a.page_table, jp, a.pps, a.max_segs, a.n_virtual, a.n_phys);
      s_phys[i] = ph;
      s_pos[i] = ph >= 0 ? jp * P : -1;
    }
    __syncthreads();

    const int nt = cn << tpp_log2;         // tiles in this chunk
    const int nsteps = (nt + 1) >> 1;
    // cooperative copy: thread t moves 16 B of K and 16 B of V of tile (t / 256)
    const int ct = tid >> 8;               // which tile of the step
    const int cb = (tid & 255) * 16;       // byte offset inside the tile (D = 128)
    auto tile_info = [&](int t, int& ph, int& pos) {
      if (t >= nt) { ph = -1; pos = -1; return; }
      const int e = t >> tpp_log2;
      ph = s_phys[e];
      pos = s_pos[e] < 0 ? -1 : s_pos[e] + (t & (tpp - 1)) * kTile;
    };
    auto load_step = [&](int st, s16x8& kx, s16x8& vx) {
      int ph, pos;
      tile_info(2 * st + ct, ph, pos);
      const s16x8 z = {0, 0, 0, 0, 0, 0, 0, 0};
      kx = z;
      vx = z;
      if (ph >= 0 && cb < TB) {
        const int64_t base = ((int64_t)ph * P + (int64_t)((2 * st + ct) & (tpp - 1)) * kTile) * D;
        kx = *reinterpret_cast<const s16x8*>(reinterpret_cast<const char*>(a.k_pool + base) + cb);
        vx = *reinterpret_cast<const s16x8*>(reinterpret_cast<const char*>(a.v_pool + base) + cb);
      }
    };
    auto store_stage = [&](int stage, const s16x8& kx, const s16x8& vx) {
      if (cb < TB) {
        *reinterpret_cast<s16x8*>(&s_kv[stage][ct * TB + cb]) = kx;
        *reinterpret_cast<s16x8*>(&s_kv[stage][2 * TB + ct * TB + cb]) = vx;
      }
    };

    s16x8 kx, vx;
    load_step(0, kx, vx);
    store_stage(0, kx, vx);
    __syncthreads();
    for (int st = 0; st < nsteps; ++st) {
      const int stage = st & 1;
      int ph0, pos0, ph1, pos1;
      tile_info(2 * st, ph0, pos0);
      tile_info(2 * st + 1, ph1, pos1);
      if (pos0 > vis_hi || (pos0 < 0 && pos1 > vis_hi)) { done = true; break; }   // block-uniform
      const bool has_next = st + 1 < nsteps;
      if (has_next) load_step(st + 1, kx, vx);

      // S^T = K . Q^T
      const char* kb = s_kv[stage];
      f32x16 sacc = {};
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const s16x8 kop = *reinterpret_cast<const s16x8*>(
            kb + (j >> 4) * TB + (((2 * s + hf) * kTile + (j & 15)) * 16));
        sacc = mfma32x32x16(kop, qreg[s], sacc);
      }
      // lane's keys: kk(rr) = 8 * (rr / 4) + 4 * hf + rr % 4 (tile kk / 16)
      const bool full = ph0 >= 0 && ph1 >= 0 && pos1 + kTile - 1 <= vis_lo;
      float sv[16];
      if (full) {
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) sv[rr] = sacc[rr];
      } else {
        const int lim = vis_row;
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int kk = 8 * (rr >> 2) + 4 * hf + (rr & 3);
          const int tp = (kk < 16 ? pos0 : pos1);
          const int p = tp + (kk & 15);
          sv[rr] = (tp >= 0 && p <= lim) ? sacc[rr] : -INFINITY;
        }
      }
      float mx = sv[0];
#pragma unroll
      for (int rr = 1; rr < 16; ++rr) mx = fmaxf(mx, sv[rr]);
      mx = fmaxf(mx, swap_halves(mx));
      const float m_new = fmaxf(m, mx);
      if (__ballot(m_new > m) != 0ull) {   // rescale only when some row's max grew
        const float alpha = (m == -INFINITY) ? 0.f : fast_exp2((m - m_new) * c);
        lsum *= alpha;
#pragma unroll
        for (int d = 0; d < NDB; ++d) acc[d] *= alpha;
        m = m_new;
      }
      const float mc = (m == -INFINITY) ? 0.f : m * c;
      float pv[16];
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        pv[rr] = fast_exp2(fmaf(sv[rr], c, -mc));
        lsum += pv[rr];
      }
      s16x8 pb[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const s16x4 lo = pack_bf16x4(pv[8 * t], pv[8 * t + 1], pv[8 * t + 2], pv[8 * t + 3]);
        const s16x4 hi = pack_bf16x4(pv[8 * t + 4], pv[8 * t + 5], pv[8 * t + 6], pv[8 * t + 7]);
        pb[t] = (s16x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      }
      // O^T += V^T . P^T; k-slot 8 hf + e of step t <-> key 16 t + (e < 4 ? 4 hf + e : 8 + 4 hf + e - 4)
      const char* vb = s_kv[stage] + 2 * TB;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int d = 0; d < NDB; ++d) {
          const int dd = d * 32 + j;
          const char* row = vb + t * TB + dd * kTile * 2;
          const s16x4 v0 = *reinterpret_cast<const s16x4*>(row + 8 * hf);
          const s16x4 v1 = *reinterpret_cast<const s16x4*>(row + 16 + 8 * hf);
          const s16x8 vop = (s16x8){v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
          acc[d] = mfma32x32x16(vop, pb[t], acc[d]);
        }
      }

      if (has_next) store_stage(stage ^ 1, kx, vx);
      __syncthreads();
    }
  }

  const float ltot = lsum + swap_halves(lsum);
  if (!row_ok) return;
  const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
  __bf16* op = a.out + ((int64_t)(q0 + qi) * a.Hq + g * G + hh) * D;
#pragma unroll
  for (int d = 0; d < NDB; ++d) {
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int dd = d * 32 + 8 * q4 + 4 * hf;
      const s16x4 o = pack_bf16x4(acc[d][4 * q4] * inv, acc[d][4 * q4 + 1] * inv,
                                  acc[d][4 * q4 + 2] * inv, acc[d][4 * q4 + 3] * inv);
      *reinterpret_cast<s16x4*>(op + dd) = o;
    }
  }
  if (hf == 0 && a.lse != nullptr)
    a.lse[(int64_t)(q0 + qi) * a.Hq + g * G + hh] =
        ltot > 0.f ? (m * c + __log2f(ltot)) * kLn2 : -INFINITY;
}

hipError_t launch_prefill(const FwdArgs& a, hipStream_t stream) {
  const dim3 grid(a.units * a.row_blocks), block(kPfThreads);
  if (a.D == 128)
    hipLaunchKernelGGL(prefill_kernel<128>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(prefill_kernel<64>, grid, block, 0, stream, a);
  return hipGetLastError();
}

int prefill_rows_per_block() { return kPfRows; }

}  // namespace segpa
