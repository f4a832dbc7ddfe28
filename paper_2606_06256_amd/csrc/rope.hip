// RoPE positional alignment of cached key pages, in place.
//
// What is computed: Section 4.2 ("RoPE-based positional alignment"). A key
// cached at offline position p_off and reused at online position p_on becomes
// R(p_on) R(p_off)^-1 K(p_off); the rotations of each plane commute, so this
// is the rotation by delta = p_on - p_off. Plane i pairs head dimension i
// with i + D/2 and turns by delta * base^(-2 i / D).
//
// A block takes as many pages as make four (token, chunk pair) items per
// thread. Each thread first loads its items: a token's pair of 8-dimension
// chunks (c, c + D/16), two 16-byte loads in the tile layout [D/8][16][8],
// consecutive threads on consecutive tokens. Meanwhile the block computes the
// (cos, sin) of each page's D/2 planes in float64 into LDS (the plane
// frequencies once per block); then every item is rotated and stored. Arithmetic
// is float64 with no contraction (each product and sum rounded as written),
// and the result is rounded once to bf16, to nearest with ties to even. The
// work is a read and a write of every listed page: HBM-bound.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace segpa {

namespace {

// float64 -> bf16 bits, to nearest with ties to even. Normal bf16 results
// come straight from the float64 fields: the top 7 mantissa bits, the round
// bit below them and the sticky OR of the rest (a carry out of the mantissa
// moves into the exponent, and into infinity past the largest value). Zeros,
// subnormal results and non-finite inputs take a slow path: round to odd into
// float32 (truncate, then set the last bit if anything was dropped), then to
// nearest-even into bf16; float32 keeps more than two extra bits, so the two
// roundings give the single correct one.
__device__ __noinline__ uint16_t f64_to_bf16_slow(double x) {
  if (x != x) return 0x7FC0;
  const float t = __double2float_rz(x);
  uint32_t u = __float_as_uint(t);
  if ((double)t != x) u |= 1u;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ uint16_t f64_to_bf16(double x) {
  const uint64_t b = (uint64_t)__double_as_longlong(x);
  const uint32_t hi = (uint32_t)(b >> 32), lo = (uint32_t)b;
  const int e = (int)((hi >> 20) & 0x7FF) - 1023 + 127;   // bf16 biased exponent
  if (e < 1 || e > 254) return f64_to_bf16_slow(x);
  uint32_t r = ((hi >> 16) & 0x8000u) | ((uint32_t)e << 7) | ((hi >> 13) & 0x7Fu);
  const uint32_t round = (hi >> 12) & 1u;
  const uint32_t sticky = (hi & 0xFFFu) | lo;
  const uint32_t lsb = r & 1u;
  r += round & ((sticky != 0u) | lsb);
  return (uint16_t)r;
}

}  // namespace

constexpr int kRopeBlock = 256;
constexpr int kRopeItems = 4;     // (token, chunk pair) items per thread and round

template <int D>
__global__ __launch_bounds__(kRopeBlock) void rope_align_kernel(const RopeArgs a, int ppb) {
#pragma clang fp contract(off)
  constexpr int H = D / 2;        // rotation planes
  constexpr int CH = D / 16;      // chunk pairs per token
  extern __shared__ double s_tab[];            // [ppb][H] cos, then [ppb][H] sin
  __shared__ double s_freq[H];
  double* s_cos = s_tab;
  double* s_sin = s_tab + ppb * H;
  const int64_t first = (int64_t)blockIdx.x * ppb;
  const int np = (int)min<int64_t>(ppb, a.n - first);
  const int per_page = a.P * CH;
  const int items = np * per_page;             // one page per block when a page exceeds a round
  const int tid = threadIdx.x;

  // one round: kRopeItems items per thread, loads first (they do not wait for
  // the table), then the rotation once the table is ready
  for (int r0 = 0; r0 < items; r0 += kRopeBlock * kRopeItems) {
    s16x8 x1[kRopeItems], x2[kRopeItems];
    s16x8* p1[kRopeItems];
    s16x8* p2[kRopeItems];
    int row[kRopeItems];                       // table row (page in block * H + 8 c), -1: none
#pragma unroll
    for (int k = 0; k < kRopeItems; ++k) {
      const int it = r0 + k * kRopeBlock + tid;
      row[k] = -1;
      p1[k] = p2[k] = nullptr;
      if (it < items) {
        const int j = it / per_page;           // page within the block
        const int w = it - j * per_page;
        const int ph = a.pages[first + j];
        if (ph >= 0 && (int64_t)ph < a.n_phys) {
          const int tok = w & (kTile - 1);
          const int c = (w / kTile) % CH;
          const int t = w / (kTile * CH);
          __bf16* base = a.k_pool + (int64_t)ph * a.P * D + (int64_t)t * kTile * D;
          p1[k] = reinterpret_cast<s16x8*>(base + (c * kTile + tok) * 8);
          p2[k] = reinterpret_cast<s16x8*>(base + ((c + CH) * kTile + tok) * 8);
          x1[k] = *p1[k];
          x2[k] = *p2[k];
          row[k] = j * H + c * 8;
        }
      }
    }
    if (r0 == 0) {
      for (int i = tid; i < H; i += kRopeBlock) s_freq[i] = pow(a.base, -(2.0 * i) / D);
      __syncthreads();
      for (int e = tid; e < np * H; e += kRopeBlock) {
        const int j = e / H;
        const double ang = (double)a.deltas[first + j] * s_freq[e - j * H];
        double sn, cs;
        sincos(ang, &sn, &cs);
        s_cos[e] = cs;
        s_sin[e] = sn;
      }
      __syncthreads();
    }
#pragma unroll
    for (int k = 0; k < kRopeItems; ++k) {
      if (row[k] < 0) continue;
      s16x8 y1, y2;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const double cs = s_cos[row[k] + e], sn = s_sin[row[k] + e];
        const double v1 = (double)bf16_bits_to_float((uint16_t)x1[k][e]);
        const double v2 = (double)bf16_bits_to_float((uint16_t)x2[k][e]);
        const double r1 = v1 * cs - v2 * sn;
        const double r2 = v2 * cs + v1 * sn;
        y1[e] = (short)f64_to_bf16(r1);
        y2[e] = (short)f64_to_bf16(r2);
      }
      *p1[k] = y1;
      *p2[k] = y2;
    }
  }
}

// Pages per block: enough for one round of kRopeItems items per thread (one
// page per block when a page alone exceeds that).
int rope_pages_per_block(int D, int P) {
  const int per_page = P * (D / 16);
  return std::max(1, kRopeBlock * kRopeItems / per_page);
}

hipError_t launch_rope_align(const RopeArgs& a, hipStream_t stream) {
  if (a.n <= 0) return hipSuccess;
  const int ppb = rope_pages_per_block(a.D, a.P);
  const dim3 grid((unsigned)((a.n + ppb - 1) / ppb)), block(kRopeBlock);
  const size_t lds = (size_t)ppb * (a.D / 2) * 2 * sizeof(double);
  if (a.D == 128)
    launch(rope_align_kernel<128>, grid, block, lds, stream, a, ppb);
  else
    launch(rope_align_kernel<64>, grid, block, lds, stream, a, ppb);
  return hipGetLastError();
}

}  // namespace segpa
