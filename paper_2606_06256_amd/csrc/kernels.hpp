// Kernel argument blocks and host-side launchers (internal to libsegpa.so).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace segpa {

// Optional dispatch timing. While the library's timing hooks are on, the host
// code sets these events (per host thread) before a launcher runs. They are
// attached to the kernel dispatch itself, so their elapsed time is the
// kernel's own execution: an event recorded beside a launch would add the
// time between that marker and the dispatch. With no events set, kernels
// launch as plain dispatches.
struct LaunchEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};
LaunchEvents& launch_events();

template <typename F, typename... Args>
inline void launch_with_events(F kernel, dim3 grid, dim3 block, size_t lds, hipStream_t s,
                               hipEvent_t start, hipEvent_t stop, Args... args) {
  if (start == nullptr && stop == nullptr)
    hipLaunchKernelGGL(kernel, grid, block, lds, s, args...);
  else
    hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)lds, s, start, stop, 0u, args...);
}

// One kernel dispatch, timed by the current launch events if any are set.
template <typename F, typename... Args>
inline void launch(F kernel, dim3 grid, dim3 block, size_t lds, hipStream_t s, Args... args) {
  const LaunchEvents ev = launch_events();
  launch_with_events(kernel, grid, block, lds, s, ev.start, ev.stop, args...);
}

constexpr int kTile = 16;       // tokens per KV tile; a page holds P / 16 tiles
constexpr int kWave = 64;
constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kLog2e = 1.44269504088896340736f;

// Forward pass (decode split-KV kernel, combine kernel, prefill kernel).
struct FwdArgs {
  const __bf16* q;            // [total_q, Hq, D]
  const int32_t* q_indptr;    // [B+1]
  const int32_t* ctx_lens;    // [B]
  const __bf16* k_pool;       // [n_phys, P*D], tile layout
  const __bf16* v_pool;
  const int32_t* seg_table;   // [B*Hkv*max_segs]
  const int32_t* page_table;  // [n_virtual]
  const int32_t* sel_indptr;  // [units+1]
  const int32_t* sel_pages;   // [sel_capacity]
  __bf16* out;                // [total_q, Hq, D]
  float* lse;                 // [total_q, Hq] or null
  float* part_o;              // workspace: [slots][16][D] normalised split outputs
  float* part_lse;            // workspace: [slots][16] base-2 LSE of each split
                              // (slots = total_waves + units * row_blocks)
  int64_t n_virtual;
  int64_t n_phys;
  int64_t sel_capacity;
  int32_t B, Hq, Hkv, G, D, P;
  int32_t tpp_log2;           // log2(P / 16)
  int32_t pps, max_segs, units, max_q_len, total_q;
  int32_t total_waves;        // decode: waves of the split-KV launch
  int32_t row_blocks;         // query-row blocks per unit: ceil(max_q_len * G / rows per block)
  float scale_log2;           // softmax scale * log2(e)
};

// RoPE alignment of cached key pages.
struct RopeArgs {
  __bf16* k_pool;             // [n_phys, P*D], tile layout, rotated in place
  const int32_t* pages;       // [n] physical page ids (outside [0, n_phys): skipped)
  const int32_t* deltas;      // [n] p_on - p_off of each page's tokens
  int64_t n;
  int64_t n_phys;
  int32_t D, P;
  double base;                // theta_i = base^(-2 i / D)
};

// Appending tokens to their pages (and refreshing page key sums).
struct AppendArgs {
  const int32_t* ctx_lens;    // [B] tokens stored before the append
  const int32_t* new_indptr;  // [B+1]
  const __bf16* k_new;        // [n_new, Hkv, D]
  const __bf16* v_new;
  const int32_t* seg_table;
  const int32_t* page_table;
  __bf16* k_pool;
  __bf16* v_pool;
  float* page_ksum;           // [n_phys, D] or null
  int64_t n_new, n_virtual, n_phys;
  int32_t B, Hkv, D, P, pps, max_segs;
};

// Page selection.
struct SelArgs {
  const int32_t* ctx_lens;
  const int32_t* q_indptr;
  const __bf16* q;
  const float* page_ksum;     // [n_phys, D] (TOPK)
  const int32_t* seg_table;
  const int32_t* page_table;
  const int8_t* head_policy;  // [Hkv] (HEAD_CLASS)
  const int32_t* budget;      // [B] (RANDOM_HASH / TOPK)
  int32_t* sel_indptr;        // [units+1]
  int32_t* sel_pages;         // [capacity]
  uint64_t* score_keys;       // workspace [units][max_pages] (TOPK)
  uint64_t seed;
  int64_t n_virtual, n_phys, capacity;
  int32_t mode, B, Hq, Hkv, G, D, P, pps, max_segs, units, max_pages, total_q;
  int32_t n_sink, window, forced_head, forced_tail;
};

struct SummaryArgs {
  const __bf16* k_pool;
  const int32_t* page_valid;
  float* page_ksum;
  int64_t n_phys;
  int32_t D, P;
};

struct ValidateArgs {
  const int32_t* ctx_lens;
  const int32_t* q_indptr;
  const int32_t* seg_table;
  const int32_t* page_table;
  const int32_t* sel_indptr;
  const int32_t* sel_pages;
  unsigned long long* result;  // [4]: per check class, smallest bad index (init ~0)
  int64_t n_virtual, n_phys, capacity;
  int32_t B, Hkv, P, pps, max_segs, max_q_len, total_q, units;
};

// Attention mass of the chunk tokens (probability pass).
struct MassArgs {
  const __bf16* q;            // [total_q, Hq, D]
  const int32_t* q_indptr;    // [B+1]
  const int32_t* ctx_lens;    // [B]
  const __bf16* k_pool;       // [n_phys, P*D], tile layout
  const int32_t* seg_table;
  const int32_t* page_table;
  const int32_t* sel_indptr;
  const int32_t* sel_pages;
  const float* lse;           // [total_q, Hq], natural log
  float* mass;                // [total_q, Hkv]
  int64_t n_virtual, n_phys, sel_capacity;
  int32_t B, Hq, Hkv, G, D, P, pps, max_segs, max_q_len, total_q;
  int32_t key_groups;         // blocks per unit: ceil(max_q_len / keys per block)
  float scale_log2;           // softmax scale * log2(e)
};

// Token selection by cumulative mass.
struct TokSelArgs {
  const int32_t* q_indptr;    // [B+1]
  const float* mass;          // [total_q, cols]
  uint8_t* keep;              // [total_q]
  int32_t* kept;              // [total_q] or null
  int32_t* keep_count;        // [B]
  float* token_mass;          // [total_q] or null
  double tau;
  int32_t recent, cols, B, total_q, max_q_len;
};

constexpr int kDecodeBlock = 256;   // 4 waves
constexpr int kSelectBlock = 512;
constexpr int kSelectKeyCache = 8192;  // candidate keys whose high halves the select kernel holds in LDS
constexpr int kSelectCand = 1024;      // radix-select candidate list in LDS

hipError_t launch_decode(const FwdArgs& a, hipStream_t stream);
hipError_t launch_rope_align(const RopeArgs& a, hipStream_t stream);
hipError_t launch_append(const AppendArgs& a, hipStream_t stream);
hipError_t launch_combine(const FwdArgs& a, hipStream_t stream);
int decode_blocks_per_cu(int D, int units);

hipError_t launch_prefill(const FwdArgs& a, hipStream_t stream);
int prefill_rows_per_block();
constexpr int kPrefillMinRows = 128;   // n_q * G at or above this runs the prefill kernel

hipError_t launch_select_scores(const SelArgs& a, hipStream_t stream);
hipError_t launch_select_fill(const SelArgs& a, hipStream_t stream);

constexpr int kTokSelMax = 16384;     // longest chunk the token selection sorts in LDS
hipError_t launch_token_mass(const MassArgs& a, hipStream_t stream);
int token_mass_keys_per_block();
hipError_t launch_select_tokens(const TokSelArgs& a, hipStream_t stream);

hipError_t launch_page_summary(const SummaryArgs& a, hipStream_t stream);
hipError_t launch_validate(const ValidateArgs& a, hipStream_t stream);

}  // namespace segpa
