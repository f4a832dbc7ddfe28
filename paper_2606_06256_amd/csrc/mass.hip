// Attention-mass token selection (SelectImportantTokens of Algorithm 1; the
// cumulative-mass rule of Section 4.4, with the keep-recent-N window of the
// sparse-FFN settings in Section 5).
//
// Two kernels.
//
// token_mass_kernel: the probability pass. For every token t of a request's
// query chunk and every KV head g it sums, over the query rows (query i, head
// h of group g) that see t, the softmax weight exp(scale q_ih . k_t - lse_ih),
// with lse the forward's log-sum-exp over the same selected pages. A token
// sees only the rows at or after it (causal), and only when its page is in
// the unit's selected list. The work is a dense contraction per unit,
//   W[rows x keys] = Q[rows x D] . K_chunk^T[D x keys],
// on the matrix cores (32x32x16 bf16). One block per (unit, 512 chunk
// tokens): the block's keys are copied from their pages into LDS once
// (16-token tiles, straight from HBM into LDS), then each wave streams its
// own tiles of 32 query rows (row = query * G + head, the layout of q) from
// HBM into registers, one tile ahead, and runs them against every key tile
// the rows can see. In the result layout each lane holds one key and 16 rows,
// so a key's column sum is a lane-local running sum per key tile; the waves'
// sums are added in a fixed order at the end. Each row of q is read once.
//
// select_tokens_kernel: one block per request. Token masses (the sum over the
// KV-head columns) are sorted by (mass descending, position ascending) in LDS
// with a bitonic network; an fp64 prefix sum in that order gives each token
// the mass of the tokens before it, and a token is kept when that is below
// tau * total. The last `recent` tokens are kept in any case.
#include "common.hpp"
#include "kernels.hpp"

namespace segpa {

typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace {

constexpr int kMassWaves = 8;
constexpr int kMassThreads = kMassWaves * 64;
constexpr int kMassKeys = 512;               // chunk tokens per block
constexpr int kMassKT = kMassKeys / 32;      // key tiles per block (one matrix-core column tile each)
constexpr int kMassTiles = kMassKeys / kTile + 1;  // 16-token pool tiles spanned by a block's keys
constexpr int kMassSel = 64;                 // page flags per block (>= kMassKeys / 16 + 1)

template <int D>
__global__ __launch_bounds__(kMassThreads, 1) void token_mass_kernel(const MassArgs a) {
  constexpr int KS = D / 16;                 // k-steps of the contraction
  constexpr int TB = kTile * D * 2;          // bytes of one 16-token K tile
  constexpr int PARTS = TB / 1024;           // 1 KB copies per tile
  __shared__ __attribute__((aligned(16))) char s_k[kMassTiles * TB];
  __shared__ __attribute__((aligned(16))) float s_nl[kMassWaves][32];
  __shared__ int s_sel[kMassSel];
  __shared__ int s_tile[kMassTiles];         // pool tile of each staged tile, -1: not attended

  // (unit, key group); the groups of one unit go to one XCD
  const int KG = a.key_groups;
  const int nblk = gridDim.x;
  const int b = blockIdx.x;
  const int v = (nblk % 8 == 0) ? (b % 8) * (nblk / 8) + b / 8 : b;
  const int u = v / KG;
  const int kg = v - u * KG;
  const int r = u / a.Hkv;
  const int g = u - r * a.Hkv;
  const int G = a.G;
  const int P = a.P;
  const int max_tokens = a.max_segs * a.pps * P;
  const int L = clampv(a.ctx_lens[r], 0, max_tokens);
  const int q0 = clampv(a.q_indptr[r], 0, a.total_q);
  const int nq = clampv(a.q_indptr[r + 1] - q0, 0, min(a.max_q_len, a.total_q - q0));
  const int K0 = kg * kMassKeys;
  if (K0 >= nq) return;                      // block-uniform
  const int K1 = min(nq, K0 + kMassKeys);
  const int base_pos = L - nq;               // position of chunk token 0 (negative only if nq > L)

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int hf = lane >> 5;
  const int j = lane & 31;

  // selected pages among those of the block's keys: the unit's list is
  // ascending, so they are among its last npg - j_lo entries
  const int npg = (L + P - 1) / P;
  const int p_lo = max(0, base_pos + K0);
  const int j_lo = p_lo / P;
  const int j_hi = max(0, base_pos + K1 - 1) / P;
  // the 16-token pool tiles holding the block's keys (floor division: the
  // first position may be negative when nq > L); their pages are translated
  // while the selection list is scanned
  const int tile0 = (base_pos + K0) >> 4;
  const int nt = ((base_pos + K1 - 1) >> 4) - tile0 + 1;
  if (tid < kMassSel) s_sel[tid] = 0;
  __syncthreads();
  int tile_id = -1;
  if (tid >= kMassThreads - kMassTiles) {    // the last threads translate, the first scan
    const int m = tid - (kMassThreads - kMassTiles);
    const int p = (tile0 + m) * kTile;
    if (m < nt && p >= 0) {
      const int ph = translate_page(a.seg_table + (int64_t)u * a.max_segs, a.page_table, p / P,
                                    a.pps, a.max_segs, a.n_virtual, a.n_phys);
      if (ph >= 0) tile_id = ph * (P / kTile) + (p % P) / kTile;
    }
  }
  {
    const int64_t cap = a.sel_capacity;
    const int64_t s0 = clampv<int64_t>(a.sel_indptr[u], 0, cap);
    const int64_t s1 = clampv<int64_t>(a.sel_indptr[u + 1], s0, cap);
    for (int64_t e = max(s0, s1 - (int64_t)(npg - j_lo)) + tid; e < s1; e += kMassThreads) {
      const int pj = a.sel_pages[e];
      if (pj >= j_lo && pj <= j_hi && pj < npg) s_sel[pj - j_lo] = 1;
    }
  }
  __syncthreads();
  if (tid >= kMassThreads - kMassTiles) {
    const int m = tid - (kMassThreads - kMassTiles);
    const int p = (tile0 + m) * kTile;
    s_tile[m] = (tile_id >= 0 && s_sel[p / P - j_lo] != 0) ? tile_id : -1;
  }
  __syncthreads();

  // rows R = i * G + hh (i = query of the chunk, hh = head in the group) see
  // chunk token k iff i >= k, i.e. R >= G * k; the block needs rows from
  // G * K0 on, in tiles of 32 rows
  const int rows = nq * G;
  const int t_lo = (G * K0) / 32;
  const int n_t = (rows + 31) / 32 - t_lo;
  const int nkt = (K1 - K0 + 31) / 32;
  // this wave's row tiles: passes of 8, alternate passes in reverse wave
  // order (later rows see more keys)
  auto tile_of = [&](int pass) { return t_lo + 8 * pass + ((pass & 1) ? kMassWaves - 1 - w : w); };
  // A operand of a row tile: lane (j, hf) holds row j, dims hf * D/2 + 8 ks .. + 7
  auto load_rows = [&](int t, s16x8 (&qa)[KS], float& l) {
    const int R = min(t * 32 + j, rows - 1);
    const int i = R / G;
    const int64_t qrow = (int64_t)(q0 + i) * a.Hq + g * G + (R - i * G);
    const __bf16* src = a.q + qrow * D + hf * (D / 2);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qa[ks] = *reinterpret_cast<const s16x8*>(src + 8 * ks);
    l = a.lse[qrow];
  };
  s16x8 qa[KS], qn[KS];
  float l_cur = 0.f, l_next = 0.f;
  int pass = 0;
  int t = tile_of(0);
  if (t - t_lo < n_t) load_rows(t, qa, l_cur);

#ifdef SEGPA_LDS_POISON
  // debug build: every key slot first holds NaN, so a read of a slot that no
  // copy filled, or one not ordered after its copy, shows up in the masses
  for (int i = tid * 16; i < (int)sizeof(s_k); i += kMassThreads * 16)
    *reinterpret_cast<s16x8*>(s_k + i) = kLdsPoison8;
  __syncthreads();
#endif
  // the block's keys into LDS, in pool order (tile m = pool tile tile0 + m);
  // tiles that are not attended are not copied (their columns are dropped)
  for (int x = w; x < nt * PARTS; x += kMassWaves) {
    const int m = x / PARTS;
    const int part = x - m * PARTS;
    const int id = s_tile[m];
    if (id >= 0)
      copy_to_lds(a.k_pool + (int64_t)id * kTile * D, TB, s_k + m * TB + part * 1024,
                  part * 1024 + lane * 16);
  }
  __builtin_amdgcn_s_waitcnt(0x0f70);        // vmcnt(0): this wave's copies (and rows) landed
  __syncthreads();

  // B operand of key tile kt: lane (j, hf) holds key K0 + 32 kt + j, dims
  // hf * D/2 + 8 ks .. + 7; in the pool tile layout [D/8][16][8] that is
  // 16 bytes at (dim block hf * KS + ks, token u) of staged tile m
  const int kpos0 = base_pos + K0 + j;
  const int boff = ((kpos0 >> 4) - tile0) * TB + (kpos0 & 15) * 16 + hf * KS * 256;
  const float sl2 = a.scale_log2;
  float acc[kMassKT];
#pragma unroll
  for (int kt = 0; kt < kMassKT; ++kt) acc[kt] = 0.f;

  while (t - t_lo < n_t) {
    const int Rt = t * 32;
    // next tile's rows in flight while this one is computed
    const int t_next = tile_of(pass + 1);
    const bool more = t_next - t_lo < n_t;
    if (more) load_rows(t_next, qn, l_next);
    // -lse * log2(e) of this tile's rows (-inf for rows past the end or
    // without a finite lse: they contribute nothing)
    {
      const bool ok = Rt + j < rows && l_cur > -INFINITY && l_cur < INFINITY;
      if (hf == 0) s_nl[w][j] = ok ? -l_cur * kLog2e : -INFINITY;
    }
    f32x4 nl[4];
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) nl[q4] = *reinterpret_cast<const f32x4*>(&s_nl[w][8 * q4 + 4 * hf]);
    // key tiles seen by some row of the tile
    const int kt_max = min(nkt - 1, ((Rt + 31) / G - K0) / 32);
    // exponentials of one key tile; result layout: lane holds key j and rows
    // 8 * (e / 4) + 4 * hf + e % 4. Four running sums keep four independent
    // exp/add chains in flight.
    auto weights = [&](const f32x16& c, int kt) {
      float s[4] = {0.f, 0.f, 0.f, 0.f};
      if (Rt >= G * (K0 + 32 * kt + 31)) {   // every row of the tile sees every key of the tile
#pragma unroll
        for (int e = 0; e < 16; ++e) s[e & 3] += fast_exp2(fmaf(c[e], sl2, nl[e / 4][e % 4]));
      } else {                               // the diagonal: row R sees key k iff R >= G * k
        const int lim = G * (K0 + 32 * kt + j) - Rt - 4 * hf;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int o = 8 * (e / 4) + e % 4;
          s[e & 3] += fast_exp2(o < lim ? -INFINITY : fmaf(c[e], sl2, nl[e / 4][e % 4]));
        }
      }
      return (s[0] + s[1]) + (s[2] + s[3]);
    };
    // key tiles in pairs: two independent product chains, interleaved, so
    // that each matrix-core step waits on the other chain's, not its own
#pragma unroll
    for (int kt = 0; kt < kMassKT; kt += 2) {
      if (kt > kt_max) continue;             // wave-uniform
      if (kt + 1 <= kt_max) {
        f32x16 c0 = {}, c1 = {};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const s16x8 b0 = *reinterpret_cast<const s16x8*>(s_k + boff + kt * 2 * TB + ks * 256);
          const s16x8 b1 = *reinterpret_cast<const s16x8*>(s_k + boff + (kt + 1) * 2 * TB + ks * 256);
          c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[ks], b0, c0, 0, 0, 0);
          c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[ks], b1, c1, 0, 0, 0);
        }
        acc[kt] += weights(c0, kt);
        acc[kt + 1] += weights(c1, kt + 1);
      } else {
        f32x16 c0 = {};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const s16x8 b0 = *reinterpret_cast<const s16x8*>(s_k + boff + kt * 2 * TB + ks * 256);
          c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[ks], b0, c0, 0, 0, 0);
        }
        acc[kt] += weights(c0, kt);
      }
    }
    ++pass;
    t = t_next;
    if (more) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qa[ks] = qn[ks];
      l_cur = l_next;
    }
  }

  // column sums: per key, both lane halves of every wave, in wave order
  __syncthreads();                           // every wave is done with the keys in LDS
  float* s_red = reinterpret_cast<float*>(s_k);
#pragma unroll
  for (int kt = 0; kt < kMassKT; ++kt) s_red[(w * kMassKT + kt) * 64 + lane] = acc[kt];
  __syncthreads();
  {
    const int kt = tid >> 5;                 // one key per thread: 16 tiles x 32
    const int k = K0 + tid;
    if (k < K1) {
      float m = 0.f;
      for (int ww = 0; ww < kMassWaves; ++ww)
        m += s_red[(ww * kMassKT + kt) * 64 + j] + s_red[(ww * kMassKT + kt) * 64 + 32 + j];
      const int pos = base_pos + k;
      const bool used = pos >= 0 && s_tile[(pos >> 4) - tile0] >= 0;
      a.mass[(int64_t)(q0 + k) * a.Hkv + g] = used ? m : 0.f;
    }
  }
}

// ---- token selection -------------------------------------------------------

constexpr int kTokBlock = 1024;

template <int CAP>
__global__ __launch_bounds__(kTokBlock) void select_tokens_kernel(const TokSelArgs a) {
  __shared__ uint64_t s_key[CAP];
  __shared__ uint8_t s_keep[CAP];
  __shared__ double s_dscan[kTokBlock / 64];
  __shared__ int s_iscan[kTokBlock / 64];
  const int r = blockIdx.x;
  const int tid = threadIdx.x;
  const int q0 = clampv(a.q_indptr[r], 0, a.total_q);
  const int n = clampv(a.q_indptr[r + 1] - q0, 0, min(min(a.max_q_len, CAP), a.total_q - q0));
  int N = 2;
  while (N < n) N <<= 1;

  // token masses (columns summed in column order, float32); a mass that is
  // not >= 0 (negative, NaN) counts as 0. Key: ~bits in the high word sorts
  // larger masses first, the position in the low word breaks ties.
  for (int t = tid; t < N; t += kTokBlock) {
    uint64_t key = ~0ull;
    if (t < n) {
      const float* row = a.mass + (int64_t)(q0 + t) * a.cols;
      float m = 0.f;
      for (int c = 0; c < a.cols; ++c) m += row[c];
      if (!(m >= 0.f)) m = 0.f;
      if (a.token_mass) a.token_mass[q0 + t] = m;
      key = ((uint64_t)(~__float_as_uint(m)) << 32) | (uint32_t)t;
      s_keep[t] = 0;
    }
    s_key[t] = key;
  }
  __syncthreads();

  // bitonic sort, ascending keys
  for (int kk = 2; kk <= N; kk <<= 1) {
    for (int j = kk >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < N / 2; i += kTokBlock) {
        const int lo = 2 * i - (i & (j - 1));
        const int hi = lo + j;
        const uint64_t x = s_key[lo], y = s_key[hi];
        const bool up = (lo & kk) == 0;
        if ((x > y) == up) {
          s_key[lo] = y;
          s_key[hi] = x;
        }
      }
      __syncthreads();
    }
  }

  // fp64 prefix of the sorted masses: thread tid owns sorted places
  // [tid * E, tid * E + E)
  const int E = (N + kTokBlock - 1) / kTokBlock;
  const int p0 = tid * E;
  auto mass_at = [&](int p) -> double { return (double)__uint_as_float(~(uint32_t)(s_key[p] >> 32)); };
  double loc = 0.0;
  for (int e = 0; e < E; ++e)
    if (p0 + e < n) loc += mass_at(p0 + e);
  double before, total;
  block_scan<kTokBlock>(loc, before, total, s_dscan);
  if (total > 0.0) {
    const double thr = a.tau * total;
    for (int e = 0; e < E && p0 + e < n; ++e) {
      if (!(before < thr)) break;
      s_keep[(uint32_t)s_key[p0 + e]] = 1;
      before += mass_at(p0 + e);
    }
  }
  __syncthreads();

  // masks, the kept rows in order, and the count
  int out = 0;
  for (int t0 = 0; t0 < n; t0 += kTokBlock) {
    const int t = t0 + tid;
    int kept = 0;
    if (t < n) {
      kept = (s_keep[t] != 0 || t >= n - a.recent) ? 1 : 0;
      a.keep[q0 + t] = (uint8_t)kept;
    }
    int ex, tot;
    block_scan<kTokBlock>(kept, ex, tot, s_iscan);
    if (kept && a.kept) a.kept[q0 + out + ex] = q0 + t;
    out += tot;
  }
  if (tid == 0) a.keep_count[r] = out;
}

}  // namespace

hipError_t launch_token_mass(const MassArgs& a, hipStream_t stream) {
  const dim3 grid((unsigned)((int64_t)a.B * a.Hkv * a.key_groups)), block(kMassThreads);
  if (a.D == 128)
    launch(token_mass_kernel<128>, grid, block, 0, stream, a);
  else
    launch(token_mass_kernel<64>, grid, block, 0, stream, a);
  return hipGetLastError();
}

int token_mass_keys_per_block() { return kMassKeys; }

hipError_t launch_select_tokens(const TokSelArgs& a, hipStream_t stream) {
  const dim3 grid(a.B), block(kTokBlock);
  if (a.max_q_len <= 1024)
    launch(select_tokens_kernel<1024>, grid, block, 0, stream, a);
  else if (a.max_q_len <= 4096)
    launch(select_tokens_kernel<4096>, grid, block, 0, stream, a);
  else
    launch(select_tokens_kernel<kTokSelMax>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace segpa
