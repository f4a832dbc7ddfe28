// RoPE positional alignment of cached key pages, in place.
//
// What is computed: Section 4.2 ("RoPE-based positional alignment"). A key
// cached at offline position p_off and reused at online position p_on becomes
// R(p_on) R(p_off)^-1 K(p_off); the rotations of each plane commute, so this
// is the rotation by delta = p_on - p_off. Plane i pairs head dimension i
// with i + D/2 and turns by delta * base^(-2 i / D).
//
// One block per listed page. The block first computes the page's D/2 (cos,
// sin) pairs in float64 into LDS; then each thread rotates one token's pair of
// 8-dimension chunks (c, c + D/16): two 16-byte loads and stores in the tile
// layout [D/8][16][8], consecutive threads on consecutive tokens. Arithmetic
// is float64 with no contraction (each product and sum rounded as written),
// and the result is rounded once to bf16, to nearest with ties to even. The
// work is a read and a write of every listed page: HBM-bound.
#include "common.hpp"
#include "kernels.hpp"

namespace segpa {

namespace {

// float64 -> bf16 bits, to nearest with ties to even: round to odd into
// float32 (truncate, then set the last bit if anything was dropped), then to
// nearest-even into bf16; float32 keeps more than two extra bits, so the two
// roundings give the single correct one.
__device__ __forceinline__ uint16_t f64_to_bf16(double x) {
  if (x != x) return 0x7FC0;
  const float t = __double2float_rz(x);
  uint32_t u = __float_as_uint(t);
  if ((double)t != x) u |= 1u;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

}  // namespace

template <int D>
__global__ __launch_bounds__(128) void rope_align_kernel(const RopeArgs a) {
#pragma clang fp contract(off)
  constexpr int H = D / 2;      // rotation planes
  constexpr int CH = D / 16;    // chunk pairs per token
  __shared__ double s_cos[H], s_sin[H];
  const int64_t idx = blockIdx.x;
  const int ph = a.pages[idx];
  if (ph < 0 || (int64_t)ph >= a.n_phys) return;   // block-uniform: skipped
  const double delta = (double)a.deltas[idx];
  for (int i = threadIdx.x; i < H; i += blockDim.x) {
    const double ang = delta * pow(a.base, -(2.0 * i) / D);
    double s, c;
    sincos(ang, &s, &c);
    s_cos[i] = c;
    s_sin[i] = s;
  }
  __syncthreads();
  __bf16* page = a.k_pool + (int64_t)ph * a.P * D;
  const int items = a.P * CH;
  for (int it = threadIdx.x; it < items; it += blockDim.x) {
    const int tok = it & (kTile - 1);
    const int c = (it / kTile) % CH;
    const int t = it / (kTile * CH);
    __bf16* base = page + (int64_t)t * kTile * D;
    s16x8* p1 = reinterpret_cast<s16x8*>(base + (c * kTile + tok) * 8);
    s16x8* p2 = reinterpret_cast<s16x8*>(base + ((c + CH) * kTile + tok) * 8);
    const s16x8 x1 = *p1;
    const s16x8 x2 = *p2;
    s16x8 y1, y2;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = c * 8 + e;
      const double v1 = (double)bf16_bits_to_float((uint16_t)x1[e]);
      const double v2 = (double)bf16_bits_to_float((uint16_t)x2[e]);
      const double r1 = v1 * s_cos[i] - v2 * s_sin[i];
      const double r2 = v2 * s_cos[i] + v1 * s_sin[i];
      y1[e] = (short)f64_to_bf16(r1);
      y2[e] = (short)f64_to_bf16(r2);
    }
    *p1 = y1;
    *p2 = y2;
  }
}

hipError_t launch_rope_align(const RopeArgs& a, hipStream_t stream) {
  if (a.n <= 0) return hipSuccess;
  const dim3 grid((unsigned)a.n), block(128);
  if (a.D == 128)
    hipLaunchKernelGGL(rope_align_kernel<128>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(rope_align_kernel<64>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace segpa
