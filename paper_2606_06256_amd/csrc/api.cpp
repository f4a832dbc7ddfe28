// Host side of libsegpa.so: argument checks, workspace sizing, launch
// configuration. Every step of the computation runs in the HIP kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <tuple>
#include <vector>

#include "kernels.hpp"
#include "segpa.h"

using namespace segpa;

// Device scratch of seg_paged_attn_fwd_noalloc (split-KV partials). Each GPU
// the library runs on holds its own copy until the process ends. In host
// code `scratch` names a host-side stand-in, never the device memory: its
// device address comes from hipGetSymbolAddress (once per device, below).
static constexpr size_t kNoAllocScratchBytes = SPA_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// ---- launch timing (opt-in measurement aid) ---------------------------------
thread_local LaunchEvents t_launch_events;
struct ProfRecord {
  const char* name;
  hipEvent_t start, stop;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<ProfRecord> g_prof;

template <class F>
hipError_t timed_launch(const char* name, hipStream_t stream, F&& launch) {
  bool on;
  {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    on = g_prof_on;
  }
  if (!on) return launch();
  hipEvent_t a, b;
  if (hipEventCreate(&a) != hipSuccess) return hipErrorUnknown;
  if (hipEventCreate(&b) != hipSuccess) {
    (void)hipEventDestroy(a);
    return hipErrorUnknown;
  }
  // the events ride on the dispatch (start and end of the kernel itself)
  LaunchEvents& ev = launch_events();
  ev.start = a;
  ev.stop = b;
  const hipError_t e = launch();
  ev.start = ev.stop = nullptr;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof.push_back({name, a, b});
  return e;
}

// ---- device facts ------------------------------------------------------------
std::mutex g_dev_mu;
std::map<std::tuple<int, int, int>, int> g_decode_waves;  // (device, D, units) -> waves

int decode_waves(int D, int units) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  const auto key = std::make_tuple(dev, D, units);
  int waves = -1;
  {
    std::lock_guard<std::mutex> lk(g_dev_mu);
    auto it = g_decode_waves.find(key);
    if (it != g_decode_waves.end()) waves = it->second;
  }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus < 1)
    return -1;
  if (waves < 0) {
    // One wave per SIMD (one block of 4 waves per compute unit), each with two
    // tiles in flight. Measured on MI355X, this beats 2 or 3 waves per SIMD
    // on every decode workload (fewer, longer stream shares: less start-up
    // per byte and fewer partials to combine). Never more than the
    // registers allow.
    waves = cus * std::min(1, decode_blocks_per_cu(D, units)) * (kDecodeBlock / kWave);
    std::lock_guard<std::mutex> lk(g_dev_mu);
    g_decode_waves[key] = waves;
  }
  return waves;
}

// ---- argument checks -----------------------------------------------------------
bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

spa_status_t check_dims(const spa_dims_t* d) {
  if (d == nullptr) return SPA_ERR_INVALID_ARG;
  if (d->num_requests < 1 || d->num_kv_heads < 1 || d->num_q_heads < 1 ||
      d->num_q_heads % d->num_kv_heads != 0 || d->pages_per_segment < 1 || d->max_segments < 1 ||
      d->max_q_len < 1 || d->total_q < 0 || d->num_virtual_pages < 0 || d->num_phys_pages < 1)
    return SPA_ERR_INVALID_ARG;
  if (d->head_dim != 64 && d->head_dim != 128) return SPA_ERR_UNSUPPORTED;
  if (d->page_size < 16 || d->page_size > 256 || !is_pow2(d->page_size)) return SPA_ERR_UNSUPPORTED;
  const int64_t units = (int64_t)d->num_requests * d->num_kv_heads;
  if (units > SPA_MAX_UNITS) return SPA_ERR_UNSUPPORTED;
  // both factors are positive int32, so max_pages < 2^62; P is a power of two,
  // so max_pages * P < 2^31 exactly when max_pages < 2^31 / P (no overflow)
  const int64_t max_pages = (int64_t)d->max_segments * d->pages_per_segment;
  if (max_pages >= (int64_t(1) << 31) / d->page_size) return SPA_ERR_UNSUPPORTED;
  if (units * max_pages >= (int64_t(1) << 31)) return SPA_ERR_UNSUPPORTED;
  if (d->num_phys_pages >= (int64_t(1) << 31) || d->num_virtual_pages >= (int64_t(1) << 31))
    return SPA_ERR_UNSUPPORTED;
  // 16-token tiles of one pool are indexed in 28 bits (1 TiB of bf16 at D = 128)
  if (d->num_phys_pages * (d->page_size / 16) >= (int64_t(1) << 28)) return SPA_ERR_UNSUPPORTED;
  if (d->num_q_heads > 4096 || (int64_t)d->total_q * d->num_q_heads >= (int64_t(1) << 31))
    return SPA_ERR_UNSUPPORTED;
  return SPA_OK;
}

int64_t units_of(const spa_dims_t* d) { return (int64_t)d->num_requests * d->num_kv_heads; }
int64_t max_pages_of(const spa_dims_t* d) { return (int64_t)d->max_segments * d->pages_per_segment; }
int row_blocks_of(const spa_dims_t* d) {
  const int64_t rows = (int64_t)d->max_q_len * (d->num_q_heads / d->num_kv_heads);
  return (int)((rows + 15) / 16);
}
int log2i(int x) {
  int l = 0;
  while ((1 << l) < x) ++l;
  return l;
}

bool is_prefill(const spa_dims_t* d) {
  return (int64_t)d->max_q_len * (d->num_q_heads / d->num_kv_heads) >= kPrefillMinRows;
}

size_t fwd_workspace(const spa_dims_t* d) {
  const int waves = decode_waves(d->head_dim, (int)units_of(d));
  if (waves < 0) return 0;
  if (is_prefill(d)) return kAlign;  // the chunked-prefill kernel keeps no split partials
  const int64_t slots = waves + units_of(d) * row_blocks_of(d);
  return align_up((size_t)slots * 16 * d->head_dim * sizeof(float)) +
         align_up((size_t)slots * 16 * sizeof(float));
}

size_t select_workspace(const spa_dims_t* d, int32_t mode) {
  if (mode == SPA_SEL_TOPK_MEANKEY) return align_up((size_t)(units_of(d) * max_pages_of(d)) * 8);
  return 0;
}

spa_status_t hip_status(hipError_t e) { return e == hipSuccess ? SPA_OK : SPA_ERR_HIP; }

// Debug switch: with SEGPA_VALIDATE set (and not "0") in the environment, the
// forward calls first run the synchronous table and list check of
// seg_paged_attn_validate (in the call's workspace) and return its
// SPA_ERR_BAD_DATA instead of launching. Read on every call (a getenv), so a
// process can switch it.
bool validate_switch_on() {
  const char* s = std::getenv("SEGPA_VALIDATE");
  return s != nullptr && s[0] != '\0' && !(s[0] == '0' && s[1] == '\0');
}

// Device address of the current GPU's scratch, looked up on the first call on
// that device (with it current) and kept per device.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

spa_status_t scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return SPA_ERR_HIP;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr)
      return SPA_ERR_HIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return SPA_OK;
}

}  // namespace

LaunchEvents& segpa::launch_events() { return t_launch_events; }

extern "C" {

size_t seg_paged_attn_workspace_size(const spa_dims_t* dims, int32_t sel_mode) {
  if (check_dims(dims) != SPA_OK) return 0;
  const size_t f = fwd_workspace(dims);
  const size_t s = select_workspace(dims, sel_mode);
  return std::max<size_t>({f, s, 64});
}

spa_status_t seg_paged_attn_select(const spa_dims_t* dims, const spa_select_params_t* params,
                                   const int32_t* ctx_lens, const void* q, const int32_t* q_indptr,
                                   const float* page_ksum, const int32_t* seg_table,
                                   const int32_t* page_table, int32_t* sel_indptr,
                                   int32_t* sel_pages, int64_t sel_capacity, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  spa_status_t st = check_dims(dims);
  if (st != SPA_OK) return st;
  if (params == nullptr || ctx_lens == nullptr || sel_indptr == nullptr || sel_pages == nullptr)
    return SPA_ERR_INVALID_ARG;
  const int mode = params->mode;
  if (mode < SPA_SEL_ALL || mode > SPA_SEL_TOPK_MEANKEY) return SPA_ERR_INVALID_ARG;
  if (mode == SPA_SEL_HEAD_CLASS &&
      (params->head_policy == nullptr || q_indptr == nullptr || params->n_sink_tokens < 0 ||
       params->window_tokens < 0))
    return SPA_ERR_INVALID_ARG;
  if ((mode == SPA_SEL_RANDOM_HASH || mode == SPA_SEL_TOPK_MEANKEY) &&
      (params->budget_pages == nullptr || params->forced_head_pages < 0 ||
       params->forced_tail_pages < 0))
    return SPA_ERR_INVALID_ARG;
  if (mode == SPA_SEL_TOPK_MEANKEY &&
      (q == nullptr || q_indptr == nullptr || page_ksum == nullptr || seg_table == nullptr ||
       page_table == nullptr))
    return SPA_ERR_INVALID_ARG;
  const int64_t units = units_of(dims);
  const int64_t max_pages = max_pages_of(dims);
  if (sel_capacity < units * max_pages) return SPA_ERR_CAPACITY;
  const size_t need = select_workspace(dims, mode);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return SPA_ERR_WORKSPACE;

  SelArgs a{};
  a.ctx_lens = ctx_lens;
  a.q_indptr = q_indptr;
  a.q = static_cast<const __bf16*>(q);
  a.page_ksum = page_ksum;
  a.seg_table = seg_table;
  a.page_table = page_table;
  a.head_policy = params->head_policy;
  a.budget = params->budget_pages;
  a.sel_indptr = sel_indptr;
  a.sel_pages = sel_pages;
  a.score_keys = static_cast<uint64_t*>(workspace);
  a.seed = params->seed;
  a.n_virtual = dims->num_virtual_pages;
  a.n_phys = dims->num_phys_pages;
  a.capacity = sel_capacity;
  a.mode = mode;
  a.B = dims->num_requests;
  a.Hq = dims->num_q_heads;
  a.Hkv = dims->num_kv_heads;
  a.G = dims->num_q_heads / dims->num_kv_heads;
  a.D = dims->head_dim;
  a.P = dims->page_size;
  a.pps = dims->pages_per_segment;
  a.max_segs = dims->max_segments;
  a.units = (int)units;
  a.max_pages = (int)max_pages;
  a.total_q = dims->total_q;
  a.n_sink = params->n_sink_tokens;
  a.window = params->window_tokens;
  a.forced_head = params->forced_head_pages;
  a.forced_tail = params->forced_tail_pages;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (mode == SPA_SEL_TOPK_MEANKEY) {
    st = hip_status(timed_launch("select_score", s, [&] { return launch_select_scores(a, s); }));
    if (st != SPA_OK) return st;
  }
  return hip_status(timed_launch("select_fill", s, [&] { return launch_select_fill(a, s); }));
}

spa_status_t seg_paged_attn_fwd(const spa_dims_t* dims, const void* q, const int32_t* q_indptr,
                                const int32_t* ctx_lens, const void* k_pool, const void* v_pool,
                                const int32_t* seg_table, const int32_t* page_table,
                                const int32_t* sel_indptr, const int32_t* sel_pages,
                                int64_t sel_capacity, void* out, float* lse, void* workspace,
                                size_t workspace_bytes, void* stream) {
  spa_status_t st = check_dims(dims);
  if (st != SPA_OK) return st;
  if (q == nullptr || q_indptr == nullptr || ctx_lens == nullptr || k_pool == nullptr ||
      v_pool == nullptr || seg_table == nullptr || page_table == nullptr || sel_indptr == nullptr ||
      sel_pages == nullptr || out == nullptr || sel_capacity < 0 ||
      sel_capacity >= (int64_t(1) << 31))
    return SPA_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(k_pool) | reinterpret_cast<uintptr_t>(v_pool) |
       reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(out)) & 15)
    return SPA_ERR_INVALID_ARG;
  const size_t need = fwd_workspace(dims);
  if (need == 0) return SPA_ERR_HIP;
  if (workspace == nullptr || workspace_bytes < need) return SPA_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) & 15) return SPA_ERR_INVALID_ARG;
  if (dims->total_q == 0) return SPA_OK;
  if (validate_switch_on()) {
    st = seg_paged_attn_validate(dims, ctx_lens, q_indptr, seg_table, page_table, sel_indptr,
                                 sel_pages, sel_capacity, nullptr, nullptr, workspace,
                                 workspace_bytes, stream);
    if (st != SPA_OK) return st;
  }

  const int units = (int)units_of(dims);
  FwdArgs a{};
  a.q = static_cast<const __bf16*>(q);
  a.q_indptr = q_indptr;
  a.ctx_lens = ctx_lens;
  a.k_pool = static_cast<const __bf16*>(k_pool);
  a.v_pool = static_cast<const __bf16*>(v_pool);
  a.seg_table = seg_table;
  a.page_table = page_table;
  a.sel_indptr = sel_indptr;
  a.sel_pages = sel_pages;
  a.out = static_cast<__bf16*>(out);
  a.lse = lse;
  a.n_virtual = dims->num_virtual_pages;
  a.n_phys = dims->num_phys_pages;
  a.sel_capacity = sel_capacity;
  a.B = dims->num_requests;
  a.Hq = dims->num_q_heads;
  a.Hkv = dims->num_kv_heads;
  a.G = dims->num_q_heads / dims->num_kv_heads;
  a.D = dims->head_dim;
  a.P = dims->page_size;
  a.tpp_log2 = log2i(dims->page_size / 16);
  a.pps = dims->pages_per_segment;
  a.max_segs = dims->max_segments;
  a.units = units;
  a.max_q_len = dims->max_q_len;
  a.total_q = dims->total_q;
  a.total_waves = decode_waves(a.D, units);
  a.row_blocks = row_blocks_of(dims);
  const float scale = dims->softmax_scale > 0.f ? dims->softmax_scale
                                                : 1.0f / std::sqrt((float)dims->head_dim);
  a.scale_log2 = scale * kLog2e;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t rows = (int64_t)dims->max_q_len * a.G;
  if (is_prefill(dims)) {
    // chunked prefill: one block per (unit, row block), all selected keys, no split
    a.row_blocks = (int)((rows + prefill_rows_per_block() - 1) / prefill_rows_per_block());
    return hip_status(timed_launch("prefill_attn", s, [&] { return launch_prefill(a, s); }));
  }
  const int64_t slots = a.total_waves + (int64_t)units * a.row_blocks;
  a.part_o = static_cast<float*>(workspace);
  a.part_lse = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                        align_up((size_t)slots * 16 * a.D * sizeof(float)));
  st = hip_status(timed_launch("decode_attn", s, [&] { return launch_decode(a, s); }));
  if (st != SPA_OK) return st;
  return hip_status(timed_launch("combine", s, [&] { return launch_combine(a, s); }));
}

spa_status_t seg_paged_attn_fwd_noalloc(const spa_dims_t* dims, const void* q,
                                        const int32_t* q_indptr, const int32_t* ctx_lens,
                                        const void* k_pool, const void* v_pool,
                                        const int32_t* seg_table, const int32_t* page_table,
                                        const int32_t* sel_indptr, const int32_t* sel_pages,
                                        int64_t sel_capacity, void* out, float* lse, void* stream) {
  const spa_status_t st = check_dims(dims);
  if (st != SPA_OK) return st;
  const size_t need = fwd_workspace(dims);
  if (need == 0) return SPA_ERR_HIP;
  if (need > kNoAllocScratchBytes) return SPA_ERR_WORKSPACE;
  void* ws = nullptr;
  const spa_status_t sst = scratch_of_current_device(&ws);
  if (sst != SPA_OK) return sst;
  // the same checks and kernels as seg_paged_attn_fwd, over the built-in scratch
  return seg_paged_attn_fwd(dims, q, q_indptr, ctx_lens, k_pool, v_pool, seg_table, page_table,
                            sel_indptr, sel_pages, sel_capacity, out, lse, ws,
                            kNoAllocScratchBytes, stream);
}

spa_status_t seg_paged_attn_page_summary(const spa_dims_t* dims, const void* k_pool,
                                         const int32_t* page_valid_tokens, float* page_ksum,
                                         void* stream) {
  const spa_status_t st = check_dims(dims);
  if (st != SPA_OK) return st;
  if (k_pool == nullptr || page_valid_tokens == nullptr || page_ksum == nullptr)
    return SPA_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(k_pool) | reinterpret_cast<uintptr_t>(page_ksum)) & 15)
    return SPA_ERR_INVALID_ARG;
  SummaryArgs a{};
  a.k_pool = static_cast<const __bf16*>(k_pool);
  a.page_valid = page_valid_tokens;
  a.page_ksum = page_ksum;
  a.n_phys = dims->num_phys_pages;
  a.D = dims->head_dim;
  a.P = dims->page_size;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return hip_status(timed_launch("page_summary", s, [&] { return launch_page_summary(a, s); }));
}

spa_status_t seg_paged_attn_append(const spa_dims_t* dims, const int32_t* ctx_lens,
                                   const int32_t* new_indptr, const void* k_new, const void* v_new,
                                   int64_t n_new, const int32_t* seg_table,
                                   const int32_t* page_table, void* k_pool, void* v_pool,
                                   float* page_ksum, void* stream) {
  const spa_status_t st = check_dims(dims);
  if (st != SPA_OK) return st;
  // n_new * Hkv < 2^27 (tiles of new tokens stay in 31 bits), tested without
  // forming the product: n_new * Hkv <= 2^27 - 1 exactly when n_new <= (2^27 - 1) / Hkv
  if (n_new < 0 || n_new > ((int64_t(1) << 27) - 1) / dims->num_kv_heads) return SPA_ERR_INVALID_ARG;
  if (n_new > 0 && (ctx_lens == nullptr || new_indptr == nullptr || k_new == nullptr ||
                    v_new == nullptr || seg_table == nullptr || page_table == nullptr ||
                    k_pool == nullptr || v_pool == nullptr))
    return SPA_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(k_pool) | reinterpret_cast<uintptr_t>(v_pool) |
       reinterpret_cast<uintptr_t>(k_new) | reinterpret_cast<uintptr_t>(v_new) |
       reinterpret_cast<uintptr_t>(page_ksum)) & 15)
    return SPA_ERR_INVALID_ARG;
  if (n_new == 0) return SPA_OK;
  AppendArgs a{};
  a.ctx_lens = ctx_lens;
  a.new_indptr = new_indptr;
  a.k_new = static_cast<const __bf16*>(k_new);
  a.v_new = static_cast<const __bf16*>(v_new);
  a.seg_table = seg_table;
  a.page_table = page_table;
  a.k_pool = static_cast<__bf16*>(k_pool);
  a.v_pool = static_cast<__bf16*>(v_pool);
  a.page_ksum = page_ksum;
  a.n_new = n_new;
  a.n_virtual = dims->num_virtual_pages;
  a.n_phys = dims->num_phys_pages;
  a.B = dims->num_requests;
  a.Hkv = dims->num_kv_heads;
  a.D = dims->head_dim;
  a.P = dims->page_size;
  a.pps = dims->pages_per_segment;
  a.max_segs = dims->max_segments;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return hip_status(timed_launch("append", s, [&] { return launch_append(a, s); }));
}

spa_status_t seg_paged_attn_rope_align(const spa_dims_t* dims, void* k_pool, const int32_t* pages,
                                       const int32_t* deltas, int64_t n, double rope_base,
                                       void* stream) {
  const spa_status_t st = check_dims(dims);
  if (st != SPA_OK) return st;
  if (n < 0 || n >= (int64_t(1) << 31) || !std::isfinite(rope_base) || rope_base <= 1.0)
    return SPA_ERR_INVALID_ARG;
  if (n > 0 && (k_pool == nullptr || pages == nullptr || deltas == nullptr)) return SPA_ERR_INVALID_ARG;
  if (reinterpret_cast<uintptr_t>(k_pool) & 15) return SPA_ERR_INVALID_ARG;
  if (n == 0) return SPA_OK;
  RopeArgs a{};
  a.k_pool = static_cast<__bf16*>(k_pool);
  a.pages = pages;
  a.deltas = deltas;
  a.n = n;
  a.n_phys = dims->num_phys_pages;
  a.D = dims->head_dim;
  a.P = dims->page_size;
  a.base = rope_base;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return hip_status(timed_launch("rope_align", s, [&] { return launch_rope_align(a, s); }));
}

spa_status_t seg_paged_attn_token_mass(const spa_dims_t* dims, const void* q,
                                       const int32_t* q_indptr, const int32_t* ctx_lens,
                                       const void* k_pool, const int32_t* seg_table,
                                       const int32_t* page_table, const int32_t* sel_indptr,
                                       const int32_t* sel_pages, int64_t sel_capacity,
                                       const float* lse, float* mass, void* stream) {
  const spa_status_t st = check_dims(dims);
  if (st != SPA_OK) return st;
  if (q == nullptr || q_indptr == nullptr || ctx_lens == nullptr || k_pool == nullptr ||
      seg_table == nullptr || page_table == nullptr || sel_indptr == nullptr ||
      sel_pages == nullptr || lse == nullptr || mass == nullptr || sel_capacity < 0 ||
      sel_capacity >= (int64_t(1) << 31))
    return SPA_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(k_pool) | reinterpret_cast<uintptr_t>(q)) & 15)
    return SPA_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(lse) | reinterpret_cast<uintptr_t>(mass)) & 3)
    return SPA_ERR_INVALID_ARG;
  if (dims->total_q == 0) return SPA_OK;
  MassArgs a{};
  a.q = static_cast<const __bf16*>(q);
  a.q_indptr = q_indptr;
  a.ctx_lens = ctx_lens;
  a.k_pool = static_cast<const __bf16*>(k_pool);
  a.seg_table = seg_table;
  a.page_table = page_table;
  a.sel_indptr = sel_indptr;
  a.sel_pages = sel_pages;
  a.lse = lse;
  a.mass = mass;
  a.n_virtual = dims->num_virtual_pages;
  a.n_phys = dims->num_phys_pages;
  a.sel_capacity = sel_capacity;
  a.B = dims->num_requests;
  a.Hq = dims->num_q_heads;
  a.Hkv = dims->num_kv_heads;
  a.G = dims->num_q_heads / dims->num_kv_heads;
  a.D = dims->head_dim;
  a.P = dims->page_size;
  a.pps = dims->pages_per_segment;
  a.max_segs = dims->max_segments;
  a.max_q_len = dims->max_q_len;
  a.total_q = dims->total_q;
  a.key_groups = (dims->max_q_len + token_mass_keys_per_block() - 1) / token_mass_keys_per_block();
  const float scale = dims->softmax_scale > 0.f ? dims->softmax_scale
                                                : 1.0f / std::sqrt((float)dims->head_dim);
  a.scale_log2 = scale * kLog2e;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return hip_status(timed_launch("token_mass", s, [&] { return launch_token_mass(a, s); }));
}

spa_status_t seg_paged_attn_select_tokens(const spa_dims_t* dims, const int32_t* q_indptr,
                                          const float* mass, int32_t mass_cols, double tau,
                                          int32_t recent, uint8_t* keep, int32_t* kept,
                                          int32_t* keep_count, float* token_mass, void* stream) {
  const spa_status_t st = check_dims(dims);
  if (st != SPA_OK) return st;
  if (q_indptr == nullptr || keep_count == nullptr || mass_cols < 1 || mass_cols > 4096 ||
      !(tau > 0.0 && tau <= 1.0) || recent < 0)
    return SPA_ERR_INVALID_ARG;
  if (dims->total_q > 0 && (mass == nullptr || keep == nullptr)) return SPA_ERR_INVALID_ARG;
  if ((int64_t)dims->total_q * mass_cols >= (int64_t(1) << 31)) return SPA_ERR_UNSUPPORTED;
  if (dims->max_q_len > kTokSelMax) return SPA_ERR_UNSUPPORTED;
  if ((reinterpret_cast<uintptr_t>(mass) | reinterpret_cast<uintptr_t>(kept) |
       reinterpret_cast<uintptr_t>(keep_count) | reinterpret_cast<uintptr_t>(token_mass)) & 3)
    return SPA_ERR_INVALID_ARG;
  TokSelArgs a{};
  a.q_indptr = q_indptr;
  a.mass = mass;
  a.keep = keep;
  a.kept = kept;
  a.keep_count = keep_count;
  a.token_mass = token_mass;
  a.tau = tau;
  a.recent = recent;
  a.cols = mass_cols;
  a.B = dims->num_requests;
  a.total_q = dims->total_q;
  a.max_q_len = dims->max_q_len;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return hip_status(timed_launch("select_tokens", s, [&] { return launch_select_tokens(a, s); }));
}

spa_status_t seg_paged_attn_validate(const spa_dims_t* dims, const int32_t* ctx_lens,
                                     const int32_t* q_indptr, const int32_t* seg_table,
                                     const int32_t* page_table, const int32_t* sel_indptr,
                                     const int32_t* sel_pages, int64_t sel_capacity,
                                     int32_t* bad_code, int64_t* bad_index, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  const spa_status_t st = check_dims(dims);
  if (st != SPA_OK) return st;
  if (ctx_lens == nullptr || q_indptr == nullptr || seg_table == nullptr || page_table == nullptr ||
      sel_indptr == nullptr || sel_pages == nullptr || sel_capacity < 0)
    return SPA_ERR_INVALID_ARG;
  if (workspace == nullptr || workspace_bytes < 64) return SPA_ERR_WORKSPACE;
  ValidateArgs a{};
  a.ctx_lens = ctx_lens;
  a.q_indptr = q_indptr;
  a.seg_table = seg_table;
  a.page_table = page_table;
  a.sel_indptr = sel_indptr;
  a.sel_pages = sel_pages;
  a.result = static_cast<unsigned long long*>(workspace);
  a.n_virtual = dims->num_virtual_pages;
  a.n_phys = dims->num_phys_pages;
  a.capacity = sel_capacity;
  a.B = dims->num_requests;
  a.Hkv = dims->num_kv_heads;
  a.P = dims->page_size;
  a.pps = dims->pages_per_segment;
  a.max_segs = dims->max_segments;
  a.max_q_len = dims->max_q_len;
  a.total_q = dims->total_q;
  a.units = (int)units_of(dims);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (hipMemsetAsync(workspace, 0xFF, 4 * sizeof(unsigned long long), s) != hipSuccess)
    return SPA_ERR_HIP;
  if (launch_validate(a, s) != hipSuccess) return SPA_ERR_HIP;
  unsigned long long res[4];
  if (hipMemcpyAsync(res, workspace, sizeof(res), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return SPA_ERR_HIP;
  for (int k = 0; k < 4; ++k) {
    if (res[k] != ~0ull) {
      if (bad_code) *bad_code = k + 1;
      if (bad_index) *bad_index = (int64_t)res[k];
      return SPA_ERR_BAD_DATA;
    }
  }
  if (bad_code) *bad_code = 0;
  if (bad_index) *bad_index = -1;
  return SPA_OK;
}

const char* seg_paged_attn_status_string(spa_status_t status) {
  // a C caller may pass any int: read the raw value rather than the enum
  int32_t code;
  std::memcpy(&code, &status, sizeof code);
  switch (code) {
    case SPA_OK: return "ok";
    case SPA_ERR_INVALID_ARG: return "invalid argument";
    case SPA_ERR_UNSUPPORTED: return "unsupported shape or parameter";
    case SPA_ERR_WORKSPACE: return "workspace missing or too small";
    case SPA_ERR_CAPACITY: return "sel_capacity below B * Hkv * max_segments * pages_per_segment";
    case SPA_ERR_HIP: return "HIP runtime error";
    case SPA_ERR_BAD_DATA: return "invalid table or page-list content";
  }
  return "unknown status";
}

spa_status_t seg_paged_attn_profile_begin(void) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& r : g_prof) {
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  g_prof.clear();
  g_prof_on = true;
  return SPA_OK;
}

int32_t seg_paged_attn_profile_end(const char** names, int32_t* launches, double* total_ms,
                                   int32_t cap) {
  std::vector<ProfRecord> recs;
  {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof_on = false;
    recs.swap(g_prof);
  }
  std::vector<const char*> kinds;
  std::vector<int32_t> cnt;
  std::vector<double> ms;
  int32_t rc = 0;
  for (auto& r : recs) {
    float t = 0.f;
    if (hipEventSynchronize(r.stop) != hipSuccess || hipEventElapsedTime(&t, r.start, r.stop) != hipSuccess)
      rc = -1;
    size_t k = 0;
    while (k < kinds.size() && std::strcmp(kinds[k], r.name) != 0) ++k;
    if (k == kinds.size()) {
      kinds.push_back(r.name);
      cnt.push_back(0);
      ms.push_back(0.0);
    }
    cnt[k] += 1;
    ms[k] += t;
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  if (rc < 0) return rc;
  const int32_t n = (int32_t)kinds.size();
  for (int32_t k = 0; k < n && k < cap; ++k) {
    if (names) names[k] = kinds[k];
    if (launches) launches[k] = cnt[k];
    if (total_ms) total_ms[k] = ms[k];
  }
  return n;
}

}  // extern "C"
