// Building head-segmented KV state: appending new tokens' keys and values to
// their pages, then refreshing the key sums of the pages that changed.
//
// What is computed: Section 4.4 (BuildState builds the reusable state of a
// chunk) over the head-segmented pages of Section 4.3. Request r's new tokens
// take positions ctx_lens[r], ctx_lens[r] + 1, ... of every KV head's stream;
// position t is slot t % P of logical page t / P, which Algorithm 2's
// Translate maps to a physical page. A token whose segment is unmapped is
// dropped. A refreshed key sum is the float32 rounding of the exact sum of the
// page's valid keys (accumulated in float64), as the page summary kernel.
//
// append_kernel: a block takes 16 consecutive new tokens of one KV head and
// all D/8 chunks; lane = token + 16 * chunk, so each store instruction writes
// 16 consecutive K slots (16 bytes each) or, per dimension, 16 consecutive V
// entries (32 bytes) of a [D][16] tile. Different tokens write different
// bytes, so no two lanes touch the same one.
// key_refresh_kernel: blocks (unit, round) over the unit's touched pages, one
// thread per (page, 8-dimension chunk).
#include "common.hpp"
#include "kernels.hpp"

namespace segpa {

// Token group of 16 consecutive new tokens x all chunks of one KV head per
// block: lane = token + 16 * chunk-in-round, so for each chunk the 16 tokens
// of a tile write 16 consecutive K slots and, per dimension, 16 consecutive
// V entries (32 bytes).
__global__ __launch_bounds__(256) void append_kernel(const AppendArgs a) {
  const int D = a.D;
  const int P = a.P;
  const int CH = D / 8;
  const int64_t i = (int64_t)blockIdx.x * kTile + (threadIdx.x & (kTile - 1));
  const int g = blockIdx.y;
  if (i >= a.n_new) return;
  // request of token i: last r with new_indptr[r] <= i
  int lo = 0, hi = a.B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if ((int64_t)a.new_indptr[mid] <= i) lo = mid; else hi = mid - 1;
  }
  const int r = lo;
  const int64_t pos = (int64_t)a.ctx_lens[r] + (i - a.new_indptr[r]);
  const int64_t max_tokens = (int64_t)a.max_segs * a.pps * P;
  if (pos < 0 || pos >= max_tokens) return;
  const int j = (int)(pos / P);
  const int slot = (int)(pos - (int64_t)j * P);
  const int32_t* seg_row = a.seg_table + ((int64_t)r * a.Hkv + g) * a.max_segs;
  const int ph = translate_page(seg_row, a.page_table, j, a.pps, a.max_segs, a.n_virtual, a.n_phys);
  if (ph < 0) return;
  const int t = slot >> 4, u = slot & (kTile - 1);
  const int64_t tile = (int64_t)ph * P * D + (int64_t)t * kTile * D;
  unsigned short* vt = reinterpret_cast<unsigned short*>(a.v_pool + tile);
  for (int c = threadIdx.x >> 4; c < CH; c += blockDim.x >> 4) {
    const int64_t src = (i * a.Hkv + g) * D + c * 8;
    *reinterpret_cast<s16x8*>(a.k_pool + tile + (c * kTile + u) * 8) =
        *reinterpret_cast<const s16x8*>(a.k_new + src);
    const s16x8 v = *reinterpret_cast<const s16x8*>(a.v_new + src);
#pragma unroll
    for (int e = 0; e < 8; ++e) vt[(c * 8 + e) * kTile + u] = (unsigned short)v[e];
  }
}

// Grid (unit, page round): thread (page slot, chunk) of each round of
// 256 / (D/8) pages of the unit's touched range; a tile's 16 keys are loaded
// before they are added.
__global__ __launch_bounds__(256) void key_refresh_kernel(const AppendArgs a) {
  const int u_id = blockIdx.x;                 // unit (r, g)
  const int r = u_id / a.Hkv;
  const int D = a.D;
  const int P = a.P;
  const int CH = D / 8;
  const int64_t n_r = (int64_t)a.new_indptr[r + 1] - a.new_indptr[r];
  if (n_r <= 0) return;
  const int64_t L0 = a.ctx_lens[r];
  const int64_t L1 = L0 + n_r;
  const int64_t max_tokens = (int64_t)a.max_segs * a.pps * P;
  if (L0 < 0 || L0 >= max_tokens) return;
  const int j0 = (int)(L0 / P);
  const int j1 = (int)((min(L1, max_tokens) - 1) / P);
  const int32_t* seg_row = a.seg_table + (int64_t)u_id * a.max_segs;
  const int per = blockDim.x / CH;             // pages per block round
  const int c = threadIdx.x % CH;
  if (threadIdx.x >= per * CH) return;
  for (int j = j0 + (int)blockIdx.y * per + (int)threadIdx.x / CH; j <= j1; j += (int)gridDim.y * per) {
    const int ph = translate_page(seg_row, a.page_table, j, a.pps, a.max_segs, a.n_virtual, a.n_phys);
    if (ph < 0) continue;
    const int valid = (int)min<int64_t>(P, L1 - (int64_t)j * P);
    const __bf16* base = a.k_pool + (int64_t)ph * P * D;
    double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int t = 0; t * kTile < valid; ++t) {
      s16x8 x[kTile];
      const __bf16* tp = base + (int64_t)t * kTile * D + c * kTile * 8;
#pragma unroll
      for (int uu = 0; uu < kTile; ++uu) x[uu] = *reinterpret_cast<const s16x8*>(tp + uu * 8);
#pragma unroll
      for (int uu = 0; uu < kTile; ++uu) {
        if (t * kTile + uu < valid) {
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[e] += (double)bf16_bits_to_float((uint16_t)x[uu][e]);
        }
      }
    }
    float* o = a.page_ksum + (int64_t)ph * D + c * 8;
    *reinterpret_cast<float4*>(o) = make_float4((float)acc[0], (float)acc[1], (float)acc[2], (float)acc[3]);
    *reinterpret_cast<float4*>(o + 4) = make_float4((float)acc[4], (float)acc[5], (float)acc[6], (float)acc[7]);
  }
}

hipError_t launch_append(const AppendArgs& a, hipStream_t stream) {
  if (a.n_new <= 0) return hipSuccess;
  const dim3 grid((unsigned)((a.n_new + kTile - 1) / kTile), (unsigned)a.Hkv);
  // timed as one call: the start event on the first dispatch, the stop event
  // on the last
  const LaunchEvents ev = launch_events();
  const bool refresh = a.page_ksum != nullptr;
  launch_with_events(append_kernel, grid, dim3(256), 0, stream, ev.start,
                     refresh ? nullptr : ev.stop, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess || !refresh) return e;
  launch_with_events(key_refresh_kernel, dim3((unsigned)(a.B * a.Hkv), 8), dim3(256), 0, stream,
                     nullptr, ev.stop, a);
  return hipGetLastError();
}

}  // namespace segpa
