// Page key sums for TOPK_MEANKEY, and the synchronous data validator.
#include "common.hpp"
#include "kernels.hpp"

namespace segpa {

// page_ksum[p][d] = float32(sum of the page's valid keys in dimension d),
// accumulated in float64. One thread per (physical page, 8-dimension chunk):
// the chunk of token u of tile t is 16 contiguous bytes at ((c * 16 + u) * 8).
__global__ __launch_bounds__(256) void page_summary_kernel(const SummaryArgs a) {
  const int D = a.D;
  const int P = a.P;
  const int chunks = D / 8;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t page = gid / chunks;
  const int c = (int)(gid - page * chunks);
  if (page >= a.n_phys) return;
  const int nv = clampv(a.page_valid[page], 0, P);
  double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  const __bf16* base = a.k_pool + page * (int64_t)P * D;
  // a tile's 16 tokens are loaded before any is added (16 loads in flight);
  // tokens past nv are read but not added. bf16 values of a page sum exactly
  // in float64, so the order of the additions does not matter.
  const int ntiles = (nv + kTile - 1) / kTile;
  for (int tile = 0; tile < ntiles; ++tile) {
    const __bf16* tp = base + (int64_t)tile * kTile * D + c * kTile * 8;
    s16x8 v[kTile];
#pragma unroll
    for (int uu = 0; uu < kTile; ++uu) v[uu] = *reinterpret_cast<const s16x8*>(tp + uu * 8);
#pragma unroll
    for (int uu = 0; uu < kTile; ++uu) {
      if (tile * kTile + uu < nv) {
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += (double)bf16_bits_to_float((uint16_t)v[uu][e]);
      }
    }
  }
  float4 lo4 = make_float4((float)acc[0], (float)acc[1], (float)acc[2], (float)acc[3]);
  float4 hi4 = make_float4((float)acc[4], (float)acc[5], (float)acc[6], (float)acc[7]);
  float* o = a.page_ksum + page * D + c * 8;
  *reinterpret_cast<float4*>(o) = lo4;
  *reinterpret_cast<float4*>(o + 4) = hi4;
}

hipError_t launch_page_summary(const SummaryArgs& a, hipStream_t stream) {
  const int64_t threads = a.n_phys * (a.D / 8);
  const int64_t blocks = (threads + 255) / 256;
  launch(page_summary_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

// Validator. result[k] keeps the smallest offending index of check class k:
//   0: q_indptr / query counts (index r)   1: ctx_lens (index r)
//   2: sel_indptr (index u)                3: selected page entries (index e)
__global__ __launch_bounds__(256) void validate_kernel(const ValidateArgs a) {
  const int u = blockIdx.x;
  const int tid = threadIdx.x;
  const int64_t max_tokens = (int64_t)a.max_segs * a.pps * a.P;
  if (u == 0) {
    for (int r = tid; r < a.B; r += blockDim.x) {
      const int q0 = a.q_indptr[r], q1 = a.q_indptr[r + 1];
      const int L = a.ctx_lens[r];
      const bool q_ok = q0 >= 0 && q1 >= q0 && q1 <= a.total_q && (q1 - q0) <= a.max_q_len &&
                        (q1 - q0) <= max(L, 0);
      if (!q_ok) atomicMin(&a.result[0], (unsigned long long)r);
      if (L < 0 || (int64_t)L > max_tokens) atomicMin(&a.result[1], (unsigned long long)r);
    }
    for (int v = tid; v < a.units; v += blockDim.x) {
      const int e0 = a.sel_indptr[v], e1 = a.sel_indptr[v + 1];
      const bool ok = (v > 0 || e0 == 0) && e1 >= e0 && (int64_t)e1 <= a.capacity;
      if (!ok) atomicMin(&a.result[2], (unsigned long long)v);
    }
  }
  const int e0 = a.sel_indptr[u], e1 = a.sel_indptr[u + 1];
  if (e0 < 0 || e1 < e0 || (int64_t)e1 > a.capacity) return;   // reported as class 2
  const int r = u / a.Hkv;
  const int L = a.ctx_lens[r];
  if (L < 0 || (int64_t)L > max_tokens) return;                 // reported as class 1
  const int npg = (L + a.P - 1) / a.P;
  const int32_t* seg_row = a.seg_table + (int64_t)u * a.max_segs;
  for (int e = e0 + tid; e < e1; e += blockDim.x) {
    const int j = a.sel_pages[e];
    bool ok = j >= 0 && j < npg && (e == e0 || a.sel_pages[e - 1] < j);
    if (ok) ok = translate_page(seg_row, a.page_table, j, a.pps, a.max_segs, a.n_virtual, a.n_phys) >= 0;
    if (!ok) atomicMin(&a.result[3], (unsigned long long)e);
  }
}

hipError_t launch_validate(const ValidateArgs& a, hipStream_t stream) {
  launch(validate_kernel, dim3(a.units), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace segpa
