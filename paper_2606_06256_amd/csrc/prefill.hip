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
// translated once per chunk of entries into LDS, and every 32 key steps each
// wave copies the next 64 steps' tile indices and flags into one register
// (lane i <-> step i), read back with v_readlane, so no LDS round trip sits
// in front of a step's loads. Keys stream in steps of 32 (two 16-token
// tiles): each thread loads its share of a step's K and V tiles three steps
// ahead into registers and stores it into one of four LDS stages. Per wave and
// step:
//   S^T[32 keys x 32 rows]  = K_step[32 x D] . Q^T       (D/16 steps, 32x32x16)
//   O^T[D x 32 rows]       += V_step^T[D x 32] . P^T     (2 x D/32, 32x32x16)
// In the S^T layout each lane holds 16 keys of one row, so the row max needs
// one cross-half swap and the running max, the sum and the rescale are
// lane-local; the 16 probabilities are, in order, the operand of the second
// product (the key order inside a step is permuted identically for V).
//
// Waves w and w + 4 share a SIMD. Waves 4..7 run half a step behind: in the
// interval between two barriers they first finish the previous step (its
// P.V product), while waves 0..3 do the vector work of the current step, so
// the matrix cores of each SIMD have one wave's products to run while the
// other wave computes exponentials.
#include "common.hpp"
#include "kernels.hpp"

namespace segpa {

typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f32x16 mfma32x32x16(s16x8 a, s16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// max of x over lanes l and l ^ 32 (v_permlane32_swap gives each lane's
// partner value in one of its two results and its own in the other)
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// value of lane l ^ 32
__device__ __forceinline__ float swap_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(__lane_id() < 32 ? r[1] : r[0]);
}

constexpr int kPfWaves = 8;
constexpr int kPfThreads = kPfWaves * 64;
constexpr int kPfRows = kPfWaves * 32;     // query rows per block
constexpr int kPfEntries = 1024;           // translated page entries held in LDS
constexpr int kPfStages = 4;               // LDS key steps
constexpr int kFlagStop = 1, kFlagFull = 2, kFlagPartial = 4;

template <int D>
__global__ __launch_bounds__(kPfThreads, 1) void prefill_kernel(const FwdArgs a) {
  constexpr int KS = D / 16;               // QK steps (16 dims each)
  constexpr int NDB = D / 32;              // 32-dim blocks of the output
  constexpr int TB = kTile * D * 2;        // bytes per tile
  constexpr int SB = 4 * TB;               // bytes per stage: K0 K1 V0 V1
  __shared__ __attribute__((aligned(16))) char s_kv[kPfStages * SB];
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
  const bool lag = w >= kPfWaves / 2;      // wave-uniform: the half-step-behind group
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

  const int64_t cap = a.sel_capacity;
  const int e0 = (int)clampv<int64_t>(a.sel_indptr[u], 0, cap);
  const int e1 = (int)clampv<int64_t>(a.sel_indptr[u + 1], 0, cap);
  const int n_e = max(0, e1 - e0);
  const int32_t* seg_row = a.seg_table + (int64_t)u * a.max_segs;
  const int tpp_log2 = a.tpp_log2;
  const int tpp = 1 << tpp_log2;
  const float c = a.scale_log2;
  const float grow_thr = 8.f / c;          // max growth (raw score units) that forces a rescale

  // The reference max m moves only when a row's max exceeds it by more than
  // 2^8 in probability; numerator and sum share the reference, so the result
  // is unchanged, and probabilities stay <= 256, far inside bf16/fp32. The
  // start value is finite and below any score: the first visible key moves it.
  float m = -1e30f;
  float mc = m * c;
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
    const int ct = tid >> 8;               // wave-uniform
    const int cb = (tid & 255) * 16;       // byte offset inside the tile (D = 128)
    auto tile_info = [&](int t, int& ph, int& pos) {
      if (t >= nt) { ph = -1; pos = -1; return; }
      const int e = t >> tpp_log2;
      ph = s_phys[e];
      pos = s_pos[e] < 0 ? -1 : s_pos[e] + (t & (tpp - 1)) * kTile;
    };
    // step table of 64 steps from tb, one int per lane: (this wave's pool
    // tile + 1) << 3 (0: unusable or past the chunk) | the step's flags (stop:
    // every key of the step and later is past the block's last query; full:
    // no masking needed; partial: this wave's tile ends past the context)
    int tb = 0, tab = 0;
    auto build_table = [&](int base) {
      tb = base;
      const int st = base + lane;
      int ph0, pos0, ph1, pos1;
      tile_info(2 * st, ph0, pos0);
      tile_info(2 * st + 1, ph1, pos1);
      const int mph = ct ? ph1 : ph0;
      const int mpos = ct ? pos1 : pos0;
      int f = mph >= 0 ? (mph * tpp + ((2 * st + ct) & (tpp - 1)) + 1) << 3 : 0;
      if (pos0 > vis_hi || (pos0 < 0 && pos1 > vis_hi)) f |= kFlagStop;
      if (ph0 >= 0 && ph1 >= 0 && pos1 + kTile - 1 <= vis_lo) f |= kFlagFull;
      if (mph >= 0 && L - mpos < kTile) f |= kFlagPartial;
      tab = f;
    };
    auto flags_of = [&](int st) { return __builtin_amdgcn_readlane(tab, st - tb); };
    auto stage = [&](int x) -> char* { return s_kv + (x & (kPfStages - 1)) * SB; };

    // unusable tiles and bytes past the tile read as zeros (zero-range descriptor)
    auto load_step = [&](int st, s16x8& kx, s16x8& vx) {
      const int tile = (int)((uint32_t)__builtin_amdgcn_readlane(tab, st - tb) >> 3) - 1;
      const int64_t base = uniform64((int64_t)(tile < 0 ? 0 : tile) * (kTile * D));
      const int range = tile >= 0 ? TB : 0;
      kx = __builtin_bit_cast(s16x8, __builtin_amdgcn_raw_buffer_load_b128(
                                         make_rsrc(a.k_pool + base, range), cb, 0, 0));
      vx = __builtin_bit_cast(s16x8, __builtin_amdgcn_raw_buffer_load_b128(
                                         make_rsrc(a.v_pool + base, range), cb, 0, 0));
    };
    // V slots past the context are stored as zeros (their probability is 0,
    // and stale contents there must not reach the sum); 16 B = tokens
    // tok0 .. tok0 + 7 of one dimension
    auto store_stage = [&](int st, const s16x8& kx, s16x8 vx) {
      if (flags_of(st) & kFlagPartial) {
        int ph, pos;
        tile_info(2 * st + ct, ph, pos);
        const int tok0 = (cb & 31) >> 1;
        const int valid = L - pos;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (tok0 + e >= valid) vx[e] = 0;
      }
      if (cb < TB) {
        char* sg = stage(st);
        *reinterpret_cast<s16x8*>(sg + ct * TB + cb) = kx;
        // V row d (16 tokens) is stored in the operand's key order: half h
        // holds tokens 4h..4h+3 and 8+4h..8+4h+3, and sits at half
        // h ^ ((d >> 3) & 1) so that one 16-byte operand read of 32 rows hits
        // distinct LDS banks. This thread holds tokens 8q..8q+7 of row d.
        const int d = cb >> 5;
        const int q = (cb >> 4) & 1;
        const int sw = (d >> 3) & 1;
        char* row = sg + 2 * TB + ct * TB + d * 32;
        const s16x4 lo = {vx[0], vx[1], vx[2], vx[3]};   // tokens 8q + 0..3 -> half 0
        const s16x4 hi = {vx[4], vx[5], vx[6], vx[7]};   // tokens 8q + 4..7 -> half 1
        *reinterpret_cast<s16x4*>(row + ((0 ^ sw) * 16) + q * 8) = lo;
        *reinterpret_cast<s16x4*>(row + ((1 ^ sw) * 16) + q * 8) = hi;
      }
    };

    auto qk = [&](int x) -> f32x16 {
      const char* kb = stage(x);
      f32x16 sacc = {};
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2) {
        const s16x8 kop = *reinterpret_cast<const s16x8*>(
            kb + (j >> 4) * TB + (((2 * s2 + hf) * kTile + (j & 15)) * 16));
        sacc = mfma32x32x16(kop, qreg[s2], sacc);
      }
      return sacc;
    };
    // start of step st: stop test, loads of step st + 3, masking, row max and
    // the (rare) rescale of everything accumulated so far
    auto pre = [&](int st, f32x16& sv, s16x8& kl, s16x8& vl) -> bool {
      const int fl = flags_of(st);
      if (fl & kFlagStop) return false;    // block-uniform
      load_step(st + 3, kl, vl);           // this set's data (step st) is already in LDS
      // lane's keys: kk(rr) = 8 * (rr / 4) + 4 * hf + rr % 4 (tile kk / 16)
      if (!(fl & kFlagFull)) {
        int ph0, pos0, ph1, pos1;
        tile_info(2 * st, ph0, pos0);
        tile_info(2 * st + 1, ph1, pos1);
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int kk = 8 * (rr >> 2) + 4 * hf + (rr & 3);
          const int tp = (kk < 16 ? pos0 : pos1);
          if (!(tp >= 0 && tp + (kk & 15) <= vis_row)) sv[rr] = -INFINITY;
        }
      }
      float mx = fmaxf(fmaxf(sv[0], sv[1]), sv[2]);
#pragma unroll
      for (int rr = 3; rr < 15; rr += 2) mx = fmaxf(fmaxf(mx, sv[rr]), sv[rr + 1]);
      mx = fmaxf(mx, sv[15]);
      const float m_new = fmaxf(m, max_halves(mx));
      if (__ballot(m_new - m > grow_thr) != 0ull) {
        const float mt = m_new - m > grow_thr ? m_new : m;
        const float alpha = fast_exp2((m - mt) * c);
        lsum *= alpha;
#pragma unroll
        for (int d = 0; d < NDB; ++d) acc[d] *= alpha;
        m = mt;
        mc = m * c;
      }
      return true;
    };
    // exponentials of step st (into pb), interleaved with the scores of step st + 1
    auto qk_exp = [&](int st, const f32x16& sv, f32x16& nxt, s16x8 (&pb)[2]) {
      float pv[16];
      const char* kb = stage(st + 1);
      f32x16 sn_acc = {};
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2) {
        const s16x8 kop = *reinterpret_cast<const s16x8*>(
            kb + (j >> 4) * TB + (((2 * s2 + hf) * kTile + (j & 15)) * 16));
        sn_acc = mfma32x32x16(kop, qreg[s2], sn_acc);
#pragma unroll
        for (int e = 0; e < 16 / KS; ++e) {
          const int rr = s2 * (16 / KS) + e;
          pv[rr] = fast_exp2(fmaf(sv[rr], c, -mc));
        }
      }
      nxt = sn_acc;
      {
        float t8[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) t8[i] = pv[i] + pv[i + 8];
        lsum += ((t8[0] + t8[4]) + (t8[1] + t8[5])) + ((t8[2] + t8[6]) + (t8[3] + t8[7]));
      }
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const s16x4 lo = pack_bf16x4(pv[8 * t], pv[8 * t + 1], pv[8 * t + 2], pv[8 * t + 3]);
        const s16x4 hi = pack_bf16x4(pv[8 * t + 4], pv[8 * t + 5], pv[8 * t + 6], pv[8 * t + 7]);
        pb[t] = (s16x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      }
    };
    // O^T += V^T . P^T for step x; k-slot 8 hf + e of tile t <-> key
    // 16 t + (e < 4 ? 4 hf + e : 8 + 4 hf + e - 4)
    auto pv_step = [&](int x, const s16x8 (&pb)[2]) {
      const char* vb = stage(x) + 2 * TB;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int d = 0; d < NDB; ++d) {
          const int dd = d * 32 + j;
          const s16x8 vop = *reinterpret_cast<const s16x8*>(
              vb + t * TB + dd * kTile * 2 + (hf ^ ((dd >> 3) & 1)) * 16);
          acc[d] = mfma32x32x16(vop, pb[t], acc[d]);
        }
      }
    };

    s16x8 kx0, vx0, kx1, vx1, kx2, vx2;
    build_table(0);
    load_step(0, kx0, vx0);
    load_step(1, kx1, vx1);
    load_step(2, kx2, vx2);
    store_stage(0, kx0, vx0);
    store_stage(1, kx1, vx1);
    __syncthreads();
    f32x16 sa = qk(0), sb = {};
    s16x8 pb[2];                           // probabilities of the step waiting for P.V

    // one step; kl: register set of step st (reloaded with st + 3), ks: set of
    // st + 2 (stored now); cur holds the scores of st, nxt receives those of
    // st + 1. Returns false once every later key is past the block's last query.
    auto body = [&](int st, s16x8& kl, s16x8& vl, const s16x8& ks, const s16x8& vs,
                    f32x16& cur, f32x16& nxt) -> bool {
      if (st > 0 && (st & 31) == 0) build_table(st);
      if (!lag) {
        if (!pre(st, cur, kl, vl)) return false;
        qk_exp(st, cur, nxt, pb);
        pv_step(st, pb);
        if (st + 2 < nsteps) store_stage(st + 2, ks, vs);
      } else {
        if (st > 0) pv_step(st - 1, pb);
        if (st + 2 < nsteps) store_stage(st + 2, ks, vs);
        if (!pre(st, cur, kl, vl)) return false;
        qk_exp(st, cur, nxt, pb);
      }
      __syncthreads();
      return true;
    };
    // register set of step x: x % 3; score buffer of step x: x % 2
    int st = 0;
    for (; st < nsteps; st += 6) {
      if (!body(st, kx0, vx0, kx2, vx2, sa, sb)) { done = true; break; }
      if (st + 1 >= nsteps) { st += 1; break; }
      if (!body(st + 1, kx1, vx1, kx0, vx0, sb, sa)) { done = true; break; }
      if (st + 2 >= nsteps) { st += 2; break; }
      if (!body(st + 2, kx2, vx2, kx1, vx1, sa, sb)) { done = true; break; }
      if (st + 3 >= nsteps) { st += 3; break; }
      if (!body(st + 3, kx0, vx0, kx2, vx2, sb, sa)) { done = true; break; }
      if (st + 4 >= nsteps) { st += 4; break; }
      if (!body(st + 4, kx1, vx1, kx0, vx0, sa, sb)) { done = true; break; }
      if (st + 5 >= nsteps) { st += 5; break; }
      if (!body(st + 5, kx2, vx2, kx1, vx1, sb, sa)) { done = true; break; }
    }
    // the lagging group still owes P.V of the chunk's last step (a stop
    // happens before a step's exponentials, so nothing is owed then)
    if (lag && !done) pv_step(nsteps - 1, pb);
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
