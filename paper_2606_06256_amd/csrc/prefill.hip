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
// tiles) through eight LDS stages: the K and V tiles of a step are copied from
// HBM straight into LDS (buffer loads with the LDS destination) six steps
// ahead, so no register staging and no LDS store instructions are needed.
// Per wave and step:
//   S^T[32 keys x 32 rows]  = K_step[32 x D] . Q^T       (D/16 steps, 32x32x16)
//   O^T[D x 32 rows]       += V_step^T[D x 32] . P^T     (2 x D/32, 32x32x16)
// In the S^T layout each lane holds 16 keys of one row, so the sum and the
// rescale are lane-local. The probabilities of a step are taken against a
// reference max that moves rarely: a step only checks that each lane's 16
// probabilities sum to at most 2^8, and only when one does not is the row max
// formed (one cross-half swap) and the reference moved to it. The probabilities of tokens 8h..8h+7 of a tile must sit in lane
// half h to meet V rows in token order. The S^T layout gives lane half h the
// key rows 4h..4h+3 and 8+4h..8+4h+3 of each 16, so key row i of the K
// operand holds the token whose index is i with bits 2 and 3 exchanged; the
// probabilities then come out in V's token order with no lane exchange.
//
// Waves w and w + 4 share a SIMD. Waves 4..7 run half a step behind: in the
// interval between two barriers they first finish the previous step (its
// P.V product), while waves 0..3 do the vector work of the current step. The
// gain is small: a product that waits for the busy matrix pipe also holds
// the SIMD's vector issue, so one wave's run of products does not overlap
// the other wave's exponentials (all waves in step time the same within
// noise). Vector work overlaps the products only where one wave interleaves
// its own, as the exponentials of step s do with the scores of step s + 1.
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

// exchange of bits 2 and 3 of a key index within its 16-token tile
__device__ __forceinline__ int swap_bits23(int i) {
  return (i & ~12) | ((i & 4) << 1) | ((i & 8) >> 1);
}

// value of lane l ^ 32
__device__ __forceinline__ float swap_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(__lane_id() < 32 ? r[1] : r[0]);
}

// Barrier of the key-step pipeline: this wave's LDS accesses are complete and
// so are its copies into LDS up to two steps ahead, while the copies of later
// steps (two per step, N in all) stay in flight. (__syncthreads would wait for
// every outstanding copy.)
template <int N>
__device__ __forceinline__ void step_barrier() {
  static_assert(N >= 0 && N < 16, "vmcnt field");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0070 | N);  // vmcnt(N) expcnt(7) lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

constexpr int kPfWaves = 8;
constexpr int kPfThreads = kPfWaves * 64;
constexpr int kPfRows = kPfWaves * 32;     // query rows per block
constexpr int kPfEntries = 1024;           // translated page entries held in LDS
constexpr int kPfStages = 8;               // LDS key steps
constexpr int kPfAhead = 6;                // steps between a copy's issue and its use
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
  const int krow = swap_bits23(j & 15);                   // token of this lane's K operand row
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

  // The reference max m moves only when a row's probabilities relative to it
  // could exceed 2^8 (then it moves to the row max); numerator and sum share
  // the reference, so the result is unchanged, and probabilities stay <= 256,
  // far inside bf16/fp32. The start value is finite and below any score: the
  // first visible key moves it.
  float m = -1e30f;
  float mc = m * c;
  float lsum = 0.f;
  f32x16 acc[NDB];
#pragma unroll
  for (int d = 0; d < NDB; ++d) acc[d] = (f32x16){};

  // LDS starts as zeros: a copy of an unusable tile (zero-range descriptor)
  // then leaves finite values behind, whatever the previous kernel left there
  for (int i = tid * 16; i < (int)sizeof(s_kv); i += kPfThreads * 16)
    *reinterpret_cast<s16x8*>(s_kv + i) = (s16x8){0, 0, 0, 0, 0, 0, 0, 0};

  const uint32_t kv_lds = __builtin_amdgcn_readfirstlane(lds_address(s_kv));
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
    // Copies: wave w moves 1 KiB of K and 1 KiB of V of tile ct = w / 4 of a
    // step (D = 64: waves with part >= 2 have nothing to move). K keeps its
    // pool layout. V row d (16 tokens, two 16-byte halves) keeps token order,
    // with half h stored at h ^ ((d >> 3) & 1) so that one operand read of 32
    // rows hits distinct LDS banks; lane l fills LDS slot part * 64 + l and so
    // reads the pool half that belongs there.
    const int ct = w >> 2;                 // wave-uniform
    const int part = w & 3;
    const bool mover = part * 1024 < TB;   // wave-uniform
    const int k_off = part * 1024 + lane * 16;
    const int v_off = [&] {
      const int slot = part * 64 + lane;
      const int d = slot >> 1;
      return d * 32 + (((slot & 1) ^ ((d >> 3) & 1)) * 16);
    }();
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
    // (rare paths take the lane index through an empty asm, so that the
    // compiler does not hoist their address arithmetic into registers that
    // stay live across the whole loop)
    auto opaque = [](int x) { asm volatile("" : "+v"(x)); return x; };
    auto build_table = [&](int base) {
      tb = base;
      const int ln = opaque(lane);
      const int st = base + ln;
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

    // HBM -> LDS copy of this wave's share of step x; unusable tiles use a
    // zero-range descriptor (no bytes are read)
    // (the addresses are scalar arithmetic on the table entry and this wave's
    // LDS slot offset, with no vector-register round trip)
    const uint32_t my_lds = __builtin_amdgcn_readfirstlane((uint32_t)(ct * TB + part * 1024));
    auto issue_copy = [&](int x) {
      if (!mover) return;
      const uint32_t ent = (uint32_t)__builtin_amdgcn_readlane(tab, x - tb);
      const int64_t tile = ent >= 8 ? (int64_t)(ent >> 3) - 1 : 0;
      const int range = ent >= 8 ? TB : 0;
      const uint32_t dst = kv_lds + (uint32_t)((x & (kPfStages - 1)) * SB) + my_lds;
#ifdef SEGPA_LDS_POISON
      // debug build: the slots this copy fills first hold NaN, so a read that
      // is not ordered after the copy's wait and barrier shows up in the output
      if (range > 0) {
        char* sl = stage(x) + ct * TB + part * 1024 + lane * 16;
        *reinterpret_cast<s16x8*>(sl) = kLdsPoison8;
        *reinterpret_cast<s16x8*>(sl + 2 * TB) = kLdsPoison8;
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      }
#endif
      copy_to_lds_at(a.k_pool + tile * (kTile * D), range, dst, k_off);
      copy_to_lds_at(a.v_pool + tile * (kTile * D), range, dst + 2 * TB, v_off);
    };
    // A tile that ends past the context: its V slots there are rewritten as
    // zeros (their probability is 0, and stale contents there must not reach
    // the sum). Runs before the barrier that publishes step x; waiting for
    // this wave's loads also orders it after the copy into the same slots.
    auto fix_partial = [&](int x) {
      if (!mover || !(flags_of(x) & kFlagPartial)) return;
      int ph, pos;
      tile_info(2 * x + ct, ph, pos);
      const int64_t base = uniform64((int64_t)(ph * tpp + ((2 * x + ct) & (tpp - 1))) * (kTile * D));
      s16x8 vx = __builtin_bit_cast(s16x8, __builtin_amdgcn_raw_buffer_load_b128(
                                               make_rsrc(a.v_pool + base, TB), v_off, 0, 0));
      const int tok0 = (v_off & 16) >> 1;  // this lane's 8 tokens start here
      const int valid = L - pos;
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (tok0 + e >= valid) vx[e] = 0;
      *reinterpret_cast<s16x8*>(stage(x) + 2 * TB + ct * TB + part * 1024 + lane * 16) = vx;
    };

    auto qk = [&](int x) -> f32x16 {
      const char* kb = stage(x);
      f32x16 sacc = {};
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2) {
        const s16x8 kop = *reinterpret_cast<const s16x8*>(
            kb + (j >> 4) * TB + (((2 * s2 + hf) * kTile + krow) * 16));
        sacc = mfma32x32x16(kop, qreg[s2], sacc);
      }
      return sacc;
    };
    // start of step st: stop test, copy of step st + kPfAhead, masking, row
    // max and the (rare) rescale of everything accumulated so far
    auto pre = [&](int st, f32x16& sv) -> bool {
      const int fl = flags_of(st);
      if (fl & kFlagStop) return false;    // block-uniform
      issue_copy(st + kPfAhead);
      // lane's keys: kk(rr) = 8 * (rr / 4) + 4 * hf + rr % 4 (tile kk / 16)
      if (!(fl & kFlagFull)) {
        int ph0, pos0, ph1, pos1;
        tile_info(2 * st, ph0, pos0);
        tile_info(2 * st + 1, ph1, pos1);
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int kk = 8 * (rr >> 2) + 4 * hf + (rr & 3);
          const int tp = (kk < 16 ? pos0 : pos1);
          if (!(tp >= 0 && tp + swap_bits23(kk & 15) <= vis_row)) sv[rr] = -INFINITY;
        }
      }
      return true;
    };
    // exponentials of step st (into pb), interleaved with the scores of step st + 1
    auto qk_exp = [&](int st, const f32x16& sv, f32x16& nxt, s16x8 (&pb)[2]) {
      float pv[16];
      __builtin_amdgcn_s_setprio(1);
      const char* kb = stage(st + 1);
      f32x16 sn_acc = {};
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2) {
        const s16x8 kop = *reinterpret_cast<const s16x8*>(
            kb + (j >> 4) * TB + (((2 * s2 + hf) * kTile + krow) * 16));
        sn_acc = mfma32x32x16(kop, qreg[s2], sn_acc);
#pragma unroll
        for (int e = 0; e < 16 / KS; ++e) {
          const int rr = s2 * (16 / KS) + e;
          pv[rr] = fast_exp2(fmaf(sv[rr], c, -mc));
        }
      }
      nxt = sn_acc;
      __builtin_amdgcn_s_setprio(0);
      auto lane_sum = [&]() {
        float t8[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) t8[i] = pv[i] + pv[i + 8];
        return ((t8[0] + t8[4]) + (t8[1] + t8[5])) + ((t8[2] + t8[6]) + (t8[3] + t8[7]));
      };
      float ps = lane_sum();
      // A lane's 16 probabilities sum to at most 2^8 unless some score exceeds
      // the reference max m by more than 8 / c (raw units); only then is the
      // row max needed. The reference then moves to the row max, everything
      // accumulated so far is rescaled, and this step's probabilities are
      // recomputed. (Not "ps <= 256" also catches the first step, where the
      // reference still holds its start value and the probabilities overflow.)
      if (__ballot(!(ps <= 256.f)) != 0ull) {
        float mx = fmaxf(fmaxf(sv[0], sv[1]), sv[2]);
#pragma unroll
        for (int rr = 3; rr < 15; rr += 2) mx = fmaxf(fmaxf(mx, sv[rr]), sv[rr + 1]);
        mx = fmaxf(mx, sv[15]);
        const float m_new = fmaxf(m, max_halves(mx));
        const float alpha = fast_exp2((m - m_new) * c);
        lsum *= alpha;
#pragma unroll
        for (int d = 0; d < NDB; ++d) acc[d] *= alpha;
        m = m_new;
        mc = m * c;
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) pv[rr] = fast_exp2(fmaf(sv[rr], c, -mc));
        ps = lane_sum();
      }
      lsum += ps;
      // tile t: pv[8 t .. 8 t + 7] are tokens 8 hf + 0..7, in order
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const s16x4 lo = pack_bf16x4(pv[8 * t], pv[8 * t + 1], pv[8 * t + 2], pv[8 * t + 3]);
        const s16x4 hi = pack_bf16x4(pv[8 * t + 4], pv[8 * t + 5], pv[8 * t + 6], pv[8 * t + 7]);
        pb[t] = (s16x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      }
    };
    // O^T += V^T . P^T for step x: k-slot 8 hf + e of tile t is token 8 hf + e
    // (the matrix-core sections of a wave run at raised issue priority, so
    // that the SIMD's other wave fills their gaps rather than delaying them)
    // The first four V operands of a step are read ahead (non-lagging waves:
    // before their score products; lagging waves: at the end of the step
    // before), so the P.V section does not start on an LDS round trip.
    constexpr int kVPre = 4;               // <= 2 * NDB for D >= 64
    s16x8 vpre[kVPre];
    auto v_operand = [&](int x, int t, int d) -> s16x8 {
      const char* vb = stage(x) + 2 * TB;
      const int dd = d * 32 + j;
      return *reinterpret_cast<const s16x8*>(vb + t * TB + dd * kTile * 2 +
                                             (hf ^ ((dd >> 3) & 1)) * 16);
    };
    auto pv_reads = [&](int x) {
#pragma unroll
      for (int i = 0; i < kVPre; ++i) vpre[i] = v_operand(x, i / NDB, i % NDB);
    };
    auto pv_step = [&](int x, const s16x8 (&pb)[2]) {
      __builtin_amdgcn_s_setprio(1);
      s16x8 vrest[2 * NDB - kVPre > 0 ? 2 * NDB - kVPre : 1];
#pragma unroll
      for (int i = kVPre; i < 2 * NDB; ++i) vrest[i - kVPre] = v_operand(x, i / NDB, i % NDB);
#pragma unroll
      for (int i = 0; i < 2 * NDB; ++i) {
        const s16x8 vop = i < kVPre ? vpre[i] : vrest[i - kVPre];
        acc[i % NDB] = mfma32x32x16(vop, pb[i / NDB], acc[i % NDB]);
      }
      // the remaining operand reads first, then the products
      if constexpr (2 * NDB > kVPre) __builtin_amdgcn_sched_group_barrier(0x100, 2 * NDB - kVPre, 0);
      __builtin_amdgcn_sched_group_barrier(0x8, 2 * NDB, 0);
      __builtin_amdgcn_s_setprio(0);
    };

    build_table(0);
#pragma unroll
    for (int x = 0; x < kPfAhead; ++x) issue_copy(x);
    fix_partial(0);
    fix_partial(1);
    step_barrier<2 * (kPfAhead - 2)>();    // steps 0 and 1 are in LDS
    f32x16 sa = qk(0), sb = {};
    s16x8 pb[2];                           // probabilities of the step waiting for P.V

    // one step; cur holds the scores of st, nxt receives those of st + 1.
    // Returns false once every later key is past the block's last query.
    auto body = [&](int st, f32x16& cur, f32x16& nxt) -> bool {
      if (st > 0 && (st & 31) == 0) build_table(st);
      if (!lag) {
        if (!pre(st, cur)) return false;
        pv_reads(st);
        qk_exp(st, cur, nxt, pb);
        pv_step(st, pb);
        fix_partial(st + 2);
      } else {
        if (st > 0) pv_step(st - 1, pb);
        fix_partial(st + 2);
        if (!pre(st, cur)) return false;
        qk_exp(st, cur, nxt, pb);
        pv_reads(st);
      }
      step_barrier<2 * (kPfAhead - 2)>();
      return true;
    };
    // score buffer of step x: x % 2
    bool stopped = false;
    for (int st = 0; st < nsteps; st += 2) {
      if (!body(st, sa, sb)) { stopped = true; break; }
      if (st + 1 >= nsteps) break;
      if (!body(st + 1, sb, sa)) { stopped = true; break; }
    }
    // the lagging group still owes P.V of the chunk's last step (a stop
    // happens before a step's exponentials, so nothing is owed then)
    if (lag && !stopped) pv_step(nsteps - 1, pb);
    done = stopped;
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);      // vmcnt(0): no copy into LDS outlives the block

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
    launch(prefill_kernel<128>, grid, block, 0, stream, a);
  else
    launch(prefill_kernel<64>, grid, block, 0, stream, a);
  return hipGetLastError();
}

int prefill_rows_per_block() { return kPfRows; }

}  // namespace segpa
