// Every status path of the C-ABI host code, run under AddressSanitizer and
// UndefinedBehaviorSanitizer with the HIP runtime and the kernel launchers
// replaced by host stand-ins. Each entry point is called with each kind of
// bad argument the header documents (and extreme sizes that would overflow
// careless integer arithmetic), then with good arguments, checking the status
// and which kernels would have been launched. Exit status 0 = all cases hold.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <string>
#include <vector>

#include "runtime_stub.hpp"
#include "segpa.h"

static int g_fail = 0;
static int g_cases = 0;

#define EXPECT(cond)                                                        \
  do {                                                                      \
    ++g_cases;                                                              \
    if (!(cond)) {                                                          \
      ++g_fail;                                                             \
      std::fprintf(stderr, "FAIL %s:%d: %s\n", __FILE__, __LINE__, #cond);  \
    }                                                                       \
  } while (0)

#define EXPECT_ST(expr, want)                                                            \
  do {                                                                                   \
    ++g_cases;                                                                           \
    const int got_ = (int)(expr);                                                        \
    if (got_ != (int)(want)) {                                                           \
      ++g_fail;                                                                          \
      std::fprintf(stderr, "FAIL %s:%d: %s -> %d, want %d\n", __FILE__, __LINE__, #expr, \
                   got_, (int)(want));                                                   \
    }                                                                                    \
  } while (0)

// Host memory standing in for device buffers: 256-byte aligned, large enough
// for every pointer the checks may look at (the stubs never read through them,
// except validate's result words).
struct Buf {
  std::vector<unsigned char> raw;
  unsigned char* p;
  explicit Buf(size_t n) : raw(n + 512) {
    p = raw.data() + (256 - reinterpret_cast<uintptr_t>(raw.data()) % 256);
  }
  void* at(size_t off = 0) { return p + off; }
};

static spa_dims_t dims(int B = 2, int Hq = 8, int Hkv = 2, int D = 128, int P = 16, int pps = 4,
                       int max_segs = 4, int max_q = 1, int total_q = 2) {
  spa_dims_t d{};
  d.num_requests = B;
  d.num_q_heads = Hq;
  d.num_kv_heads = Hkv;
  d.head_dim = D;
  d.page_size = P;
  d.pages_per_segment = pps;
  d.max_segments = max_segs;
  d.max_q_len = max_q;
  d.total_q = total_q;
  d.num_virtual_pages = 64;
  d.num_phys_pages = 64;
  d.softmax_scale = 0.f;
  return d;
}

static bool launched(std::initializer_list<const char*> want) {
  if (stub::launches.size() != want.size()) return false;
  size_t i = 0;
  for (const char* w : want)
    if (stub::launches[i++] != w) return false;
  return true;
}

static void reset() {
  stub::launches.clear();
  stub::launch_result = hipSuccess;
  stub::validate_reports_bad = false;
}

static Buf mem(1 << 22);
static void* A = mem.at(0);                         // 256-aligned
static void* A2 = mem.at(4096);
static void* MIS16 = mem.at(8);                     // 8-aligned, not 16
static void* MIS4 = mem.at(2);                      // 2-aligned
static const int32_t* I32 = static_cast<const int32_t*>(mem.at(8192));

static void check_dims_paths() {
  const int32_t cap = 1 << 20;
  spa_select_params_t prm{};
  prm.mode = SPA_SEL_ALL;
  auto sel = [&](const spa_dims_t* d) {
    return seg_paged_attn_select(d, &prm, I32, A, I32, nullptr, I32, I32, (int32_t*)A,
                                 (int32_t*)A2, cap, nullptr, 0, nullptr);
  };
  EXPECT_ST(sel(nullptr), SPA_ERR_INVALID_ARG);
  struct Case {
    spa_dims_t d;
    int want;
  };
  std::vector<Case> cases;
  auto add = [&](spa_dims_t d, int want) { cases.push_back({d, want}); };
  spa_dims_t d;
  d = dims(); d.num_requests = 0; add(d, SPA_ERR_INVALID_ARG);
  d = dims(); d.num_requests = -5; add(d, SPA_ERR_INVALID_ARG);
  d = dims(); d.num_kv_heads = 0; add(d, SPA_ERR_INVALID_ARG);
  d = dims(); d.num_q_heads = 0; add(d, SPA_ERR_INVALID_ARG);
  d = dims(); d.num_q_heads = 6; d.num_kv_heads = 4; add(d, SPA_ERR_INVALID_ARG);
  d = dims(); d.pages_per_segment = 0; add(d, SPA_ERR_INVALID_ARG);
  d = dims(); d.max_segments = 0; add(d, SPA_ERR_INVALID_ARG);
  d = dims(); d.max_q_len = 0; add(d, SPA_ERR_INVALID_ARG);
  d = dims(); d.total_q = -1; add(d, SPA_ERR_INVALID_ARG);
  d = dims(); d.num_virtual_pages = -1; add(d, SPA_ERR_INVALID_ARG);
  d = dims(); d.num_phys_pages = 0; add(d, SPA_ERR_INVALID_ARG);
  d = dims(); d.head_dim = 96; add(d, SPA_ERR_UNSUPPORTED);
  d = dims(); d.head_dim = 256; add(d, SPA_ERR_UNSUPPORTED);
  d = dims(); d.page_size = 8; add(d, SPA_ERR_UNSUPPORTED);
  d = dims(); d.page_size = 24; add(d, SPA_ERR_UNSUPPORTED);
  d = dims(); d.page_size = 512; add(d, SPA_ERR_UNSUPPORTED);
  d = dims(); d.num_requests = 2000; d.num_kv_heads = 8; d.num_q_heads = 8; add(d, SPA_ERR_UNSUPPORTED);
  // sizes chosen to overflow 32-bit (and careless 64-bit) products
  const int32_t big = std::numeric_limits<int32_t>::max();
  d = dims(); d.max_segments = big; d.pages_per_segment = big; add(d, SPA_ERR_UNSUPPORTED);
  d = dims(); d.max_segments = 1 << 16; d.pages_per_segment = 1 << 11; add(d, SPA_ERR_UNSUPPORTED);
  d = dims(8192, 8192, 8192); d.max_segments = 1 << 10; d.pages_per_segment = 1 << 10; add(d, SPA_ERR_UNSUPPORTED);
  d = dims(); d.num_phys_pages = int64_t(1) << 31; add(d, SPA_ERR_UNSUPPORTED);
  d = dims(); d.num_phys_pages = std::numeric_limits<int64_t>::max(); add(d, SPA_ERR_UNSUPPORTED);
  d = dims(); d.num_virtual_pages = std::numeric_limits<int64_t>::max(); add(d, SPA_ERR_UNSUPPORTED);
  d = dims(); d.num_phys_pages = int64_t(1) << 28; add(d, SPA_ERR_UNSUPPORTED);
  d = dims(); d.num_phys_pages = int64_t(1) << 24; d.page_size = 256; add(d, SPA_ERR_UNSUPPORTED);
  d = dims(); d.num_q_heads = 8192; d.num_kv_heads = 2; add(d, SPA_ERR_UNSUPPORTED);
  d = dims(); d.total_q = big; d.num_q_heads = 64; d.num_kv_heads = 8; add(d, SPA_ERR_UNSUPPORTED);
  d = dims(); d.num_requests = big; d.num_kv_heads = big; d.num_q_heads = big; add(d, SPA_ERR_UNSUPPORTED);
  for (const auto& c : cases) {
    reset();
    EXPECT_ST(sel(&c.d), c.want);
    EXPECT(stub::launches.empty());
    EXPECT(seg_paged_attn_workspace_size(&c.d, SPA_SEL_ALL) == 0);
  }
  d = dims();
  EXPECT(seg_paged_attn_workspace_size(&d, SPA_SEL_ALL) >= 64);
  EXPECT(seg_paged_attn_workspace_size(nullptr, SPA_SEL_ALL) == 0);
  // the TOPK rule adds one 64-bit key per candidate page
  d = dims(32, 64, 8, 128, 32, 256, 16);
  EXPECT(seg_paged_attn_workspace_size(&d, SPA_SEL_TOPK_MEANKEY) >= (size_t)32 * 8 * 16 * 256 * 8);
}

static void select_paths() {
  spa_dims_t d = dims();
  const int64_t need_cap = 2 * 2 * 4 * 4;
  spa_select_params_t p{};
  auto sel = [&](const spa_select_params_t* pp, int64_t cap = 1 << 20, void* ws = nullptr,
                 size_t wsb = 0, const int32_t* ctx = I32, const void* q = A,
                 const int32_t* qi = I32, const float* ks = (const float*)A2,
                 int32_t* ind = (int32_t*)A) {
    return seg_paged_attn_select(&d, pp, ctx, q, qi, ks, I32, I32, ind, (int32_t*)A2, cap, ws, wsb,
                                 nullptr);
  };
  reset();
  EXPECT_ST(sel(nullptr), SPA_ERR_INVALID_ARG);
  p.mode = SPA_SEL_ALL;
  EXPECT_ST(sel(&p, 1 << 20, nullptr, 0, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(sel(&p, 1 << 20, nullptr, 0, I32, A, I32, nullptr, nullptr), SPA_ERR_INVALID_ARG);
  p.mode = 7;
  EXPECT_ST(sel(&p), SPA_ERR_INVALID_ARG);
  p.mode = -1;
  EXPECT_ST(sel(&p), SPA_ERR_INVALID_ARG);
  p.mode = SPA_SEL_HEAD_CLASS;
  p.head_policy = nullptr;
  EXPECT_ST(sel(&p), SPA_ERR_INVALID_ARG);
  p.head_policy = (const int8_t*)A;
  p.n_sink_tokens = -1;
  EXPECT_ST(sel(&p), SPA_ERR_INVALID_ARG);
  p.n_sink_tokens = 4;
  p.window_tokens = -3;
  EXPECT_ST(sel(&p), SPA_ERR_INVALID_ARG);
  p.window_tokens = 256;
  EXPECT_ST(sel(&p, 1 << 20, nullptr, 0, I32, A, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT(stub::launches.empty());
  EXPECT_ST(sel(&p), SPA_OK);
  EXPECT(launched({"select_fill"}));
  for (int mode : {SPA_SEL_RANDOM_HASH, SPA_SEL_TOPK_MEANKEY}) {
    reset();
    p = spa_select_params_t{};
    p.mode = mode;
    EXPECT_ST(sel(&p), SPA_ERR_INVALID_ARG);  // no budgets
    p.budget_pages = I32;
    p.forced_head_pages = -1;
    EXPECT_ST(sel(&p), SPA_ERR_INVALID_ARG);
    p.forced_head_pages = 0;
    p.forced_tail_pages = -1;
    EXPECT_ST(sel(&p), SPA_ERR_INVALID_ARG);
    p.forced_tail_pages = 1;
    EXPECT(stub::launches.empty());
  }
  // TOPK reads q, q_indptr, the key sums and both tables
  p.mode = SPA_SEL_TOPK_MEANKEY;
  const size_t ws = seg_paged_attn_workspace_size(&d, SPA_SEL_TOPK_MEANKEY);
  EXPECT_ST(sel(&p, 1 << 20, A2, ws, I32, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(sel(&p, 1 << 20, A2, ws, I32, A, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(sel(&p, 1 << 20, A2, ws, I32, A, I32, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(seg_paged_attn_select(&d, &p, I32, A, I32, (const float*)A2, nullptr, I32, (int32_t*)A,
                                  (int32_t*)A2, 1 << 20, A2, ws, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(seg_paged_attn_select(&d, &p, I32, A, I32, (const float*)A2, I32, nullptr, (int32_t*)A,
                                  (int32_t*)A2, 1 << 20, A2, ws, nullptr), SPA_ERR_INVALID_ARG);
  // capacity and workspace
  EXPECT_ST(sel(&p, need_cap - 1, A2, ws), SPA_ERR_CAPACITY);
  EXPECT_ST(sel(&p, -1, A2, ws), SPA_ERR_CAPACITY);
  EXPECT_ST(sel(&p, need_cap, nullptr, ws), SPA_ERR_WORKSPACE);
  // one 64-bit key per candidate page (64 pages here) does not fit in 8 bytes
  EXPECT_ST(sel(&p, need_cap, A2, 8), SPA_ERR_WORKSPACE);
  EXPECT(stub::launches.empty());
  EXPECT_ST(sel(&p, need_cap, A2, ws), SPA_OK);
  EXPECT(launched({"select_score", "select_fill"}));
  // a failed launch is reported, and nothing after it is launched
  reset();
  stub::launch_result = hipErrorLaunchFailure;
  EXPECT_ST(sel(&p, need_cap, A2, ws), SPA_ERR_HIP);
  EXPECT(launched({"select_score"}));
  reset();
  p.mode = SPA_SEL_RANDOM_HASH;
  EXPECT_ST(sel(&p, need_cap), SPA_OK);       // no workspace needed
  EXPECT(launched({"select_fill"}));
}

static void fwd_paths() {
  spa_dims_t d = dims();
  const size_t ws = seg_paged_attn_workspace_size(&d, SPA_SEL_ALL);
  EXPECT(ws > 0);
  Buf wsb(ws + 64);
  void* W = wsb.at();
  struct Ptrs {
    const void *q = A, *k = A, *v = A2;
    const int32_t *qi = I32, *ctx = I32, *seg = I32, *pt = I32, *ind = I32, *pages = I32;
    void* out = A2;
    float* lse = (float*)A;
    int64_t cap = 1 << 20;
    void* ws;
    size_t wsb;
  };
  auto call = [&](const spa_dims_t& dd, const Ptrs& x) {
    return seg_paged_attn_fwd(&dd, x.q, x.qi, x.ctx, x.k, x.v, x.seg, x.pt, x.ind, x.pages, x.cap,
                              x.out, x.lse, x.ws, x.wsb, nullptr);
  };
  Ptrs ok;
  ok.ws = W;
  ok.wsb = ws;
  reset();
  {
    Ptrs x = ok; x.q = nullptr; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.qi = nullptr; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.ctx = nullptr; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.k = nullptr; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.v = nullptr; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.seg = nullptr; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.pt = nullptr; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.ind = nullptr; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.pages = nullptr; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.out = nullptr; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.cap = -1; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.cap = int64_t(1) << 31; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.k = MIS16; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.v = MIS16; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.q = MIS16; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.out = MIS16; EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    x = ok; x.ws = nullptr; EXPECT_ST(call(d, x), SPA_ERR_WORKSPACE);
    x = ok; x.wsb = ws - 1; EXPECT_ST(call(d, x), SPA_ERR_WORKSPACE);
    x = ok; x.ws = wsb.at(8); EXPECT_ST(call(d, x), SPA_ERR_INVALID_ARG);
    spa_dims_t bad = d; bad.head_dim = 80; EXPECT_ST(call(bad, ok), SPA_ERR_UNSUPPORTED);
    EXPECT(stub::launches.empty());
  }
  // no rows: nothing to launch
  spa_dims_t d0 = d;
  d0.total_q = 0;
  EXPECT_ST(call(d0, ok), SPA_OK);
  EXPECT(stub::launches.empty());
  // NULL lse is allowed
  Ptrs nl = ok;
  nl.lse = nullptr;
  EXPECT_ST(call(d, nl), SPA_OK);
  EXPECT(launched({"decode_attn", "combine"}));
  // decode rows below the prefill threshold: split-KV decode + combine
  reset();
  EXPECT_ST(call(d, ok), SPA_OK);
  EXPECT(launched({"decode_attn", "combine"}));
  // a failed decode launch stops the call before the combine
  reset();
  stub::launch_result = hipErrorLaunchFailure;
  EXPECT_ST(call(d, ok), SPA_ERR_HIP);
  EXPECT(launched({"decode_attn"}));
  // a chunk of max_q_len * G >= 128 rows takes the chunked-prefill kernel
  reset();
  spa_dims_t dp = dims(2, 8, 2, 128, 16, 4, 4, 32, 64);
  const size_t wsp = seg_paged_attn_workspace_size(&dp, SPA_SEL_ALL);
  Buf wpb(wsp + 64);
  Ptrs pp = ok;
  pp.ws = wpb.at();
  pp.wsb = wsp;
  EXPECT_ST(call(dp, pp), SPA_OK);
  EXPECT(launched({"prefill_attn"}));
  // one row fewer than the threshold stays on the decode kernel
  reset();
  spa_dims_t dd = dims(2, 8, 2, 128, 16, 4, 4, 31, 62);
  const size_t wsd = seg_paged_attn_workspace_size(&dd, SPA_SEL_ALL);
  Buf wdb(wsd + 64);
  Ptrs pd = ok;
  pd.ws = wdb.at();
  pd.wsb = wsd;
  EXPECT_ST(call(dd, pd), SPA_OK);
  EXPECT(launched({"decode_attn", "combine"}));
}

static void summary_append_rope_paths() {
  spa_dims_t d = dims();
  reset();
  EXPECT_ST(seg_paged_attn_page_summary(&d, nullptr, I32, (float*)A, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(seg_paged_attn_page_summary(&d, A, nullptr, (float*)A, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(seg_paged_attn_page_summary(&d, A, I32, nullptr, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(seg_paged_attn_page_summary(&d, MIS16, I32, (float*)A, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(seg_paged_attn_page_summary(&d, A, I32, (float*)MIS16, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT(stub::launches.empty());
  EXPECT_ST(seg_paged_attn_page_summary(&d, A, I32, (float*)A2, nullptr), SPA_OK);
  EXPECT(launched({"page_summary"}));

  auto app = [&](int64_t n, const int32_t* ctx = I32, const void* kn = A, void* kp = A,
                 float* ks = nullptr) {
    return seg_paged_attn_append(&d, ctx, I32, kn, A2, n, I32, I32, kp, A2, ks, nullptr);
  };
  reset();
  EXPECT_ST(app(-1), SPA_ERR_INVALID_ARG);
  EXPECT_ST(app(std::numeric_limits<int64_t>::max()), SPA_ERR_INVALID_ARG);
  EXPECT_ST(app(int64_t(1) << 30), SPA_ERR_INVALID_ARG);
  EXPECT_ST(app(4, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(app(4, I32, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(app(4, I32, A, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(app(4, I32, A, MIS16), SPA_ERR_INVALID_ARG);
  EXPECT_ST(app(4, I32, MIS16), SPA_ERR_INVALID_ARG);
  EXPECT_ST(app(4, I32, A, A, (float*)MIS4), SPA_ERR_INVALID_ARG);
  EXPECT(stub::launches.empty());
  EXPECT_ST(seg_paged_attn_append(&d, nullptr, nullptr, nullptr, nullptr, 0, nullptr, nullptr,
                                  nullptr, nullptr, nullptr, nullptr), SPA_OK);
  EXPECT(stub::launches.empty());
  EXPECT_ST(app(4, I32, A, A, (float*)A2), SPA_OK);
  EXPECT(launched({"append"}));

  auto rope = [&](int64_t n, double base, void* kp = A, const int32_t* pg = I32) {
    return seg_paged_attn_rope_align(&d, kp, pg, I32, n, base, nullptr);
  };
  reset();
  EXPECT_ST(rope(-1, 1e4), SPA_ERR_INVALID_ARG);
  EXPECT_ST(rope(int64_t(1) << 31, 1e4), SPA_ERR_INVALID_ARG);
  EXPECT_ST(rope(4, 1.0), SPA_ERR_INVALID_ARG);
  EXPECT_ST(rope(4, -2.0), SPA_ERR_INVALID_ARG);
  EXPECT_ST(rope(4, std::nan("")), SPA_ERR_INVALID_ARG);
  EXPECT_ST(rope(4, HUGE_VAL), SPA_ERR_INVALID_ARG);
  EXPECT_ST(rope(4, 1e4, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(rope(4, 1e4, A, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(rope(4, 1e4, MIS16), SPA_ERR_INVALID_ARG);
  EXPECT(stub::launches.empty());
  EXPECT_ST(seg_paged_attn_rope_align(&d, nullptr, nullptr, nullptr, 0, 1e4, nullptr), SPA_OK);
  EXPECT(stub::launches.empty());
  EXPECT_ST(rope(4, 1e4), SPA_OK);
  EXPECT(launched({"rope_align"}));
}

static void token_paths() {
  spa_dims_t d = dims();
  auto tm = [&](const spa_dims_t& dd, const void* q = A, const void* kp = A, const float* lse = (const float*)A,
                float* mass = (float*)A2, int64_t cap = 1 << 10) {
    return seg_paged_attn_token_mass(&dd, q, I32, I32, kp, I32, I32, I32, I32, cap, lse, mass, nullptr);
  };
  reset();
  EXPECT_ST(tm(d, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(tm(d, A, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(tm(d, A, A, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(tm(d, A, A, (const float*)A, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(tm(d, A, A, (const float*)A, (float*)A2, -1), SPA_ERR_INVALID_ARG);
  EXPECT_ST(tm(d, A, A, (const float*)A, (float*)A2, int64_t(1) << 31), SPA_ERR_INVALID_ARG);
  EXPECT_ST(tm(d, MIS16), SPA_ERR_INVALID_ARG);
  EXPECT_ST(tm(d, A, MIS16), SPA_ERR_INVALID_ARG);
  EXPECT_ST(tm(d, A, A, (const float*)MIS4), SPA_ERR_INVALID_ARG);
  EXPECT_ST(tm(d, A, A, (const float*)A, (float*)MIS4), SPA_ERR_INVALID_ARG);
  spa_dims_t bad = d;
  bad.head_dim = 96;
  EXPECT_ST(tm(bad), SPA_ERR_UNSUPPORTED);
  spa_dims_t d0 = d;
  d0.total_q = 0;
  EXPECT_ST(tm(d0), SPA_OK);
  EXPECT(stub::launches.empty());
  EXPECT_ST(tm(d), SPA_OK);
  EXPECT(launched({"token_mass"}));

  auto st = [&](const spa_dims_t& dd, int cols = 2, double tau = 0.5, int recent = 0,
                const int32_t* qi = I32, const float* mass = (const float*)A, uint8_t* keep = (uint8_t*)A2,
                int32_t* cnt = (int32_t*)A2, float* tmass = nullptr) {
    return seg_paged_attn_select_tokens(&dd, qi, mass, cols, tau, recent, keep, nullptr, cnt, tmass,
                                        nullptr);
  };
  reset();
  EXPECT_ST(st(d, 2, 0.5, 0, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(st(d, 2, 0.5, 0, I32, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(st(d, 2, 0.5, 0, I32, (const float*)A, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(st(d, 2, 0.5, 0, I32, (const float*)A, (uint8_t*)A2, nullptr), SPA_ERR_INVALID_ARG);
  for (double tau : {0.0, -0.5, 1.5, std::nan(""), HUGE_VAL}) EXPECT_ST(st(d, 2, tau), SPA_ERR_INVALID_ARG);
  EXPECT_ST(st(d, 2, 0.5, -1), SPA_ERR_INVALID_ARG);
  EXPECT_ST(st(d, 0), SPA_ERR_INVALID_ARG);
  EXPECT_ST(st(d, 4097), SPA_ERR_INVALID_ARG);
  EXPECT_ST(st(d, 2, 0.5, 0, I32, (const float*)A, (uint8_t*)A2, (int32_t*)A2, (float*)MIS4),
            SPA_ERR_INVALID_ARG);
  EXPECT_ST(st(d, 2, 0.5, 0, I32, (const float*)MIS4), SPA_ERR_INVALID_ARG);
  spa_dims_t lq = d;
  lq.max_q_len = 16385;
  EXPECT_ST(st(lq), SPA_ERR_UNSUPPORTED);
  spa_dims_t wide = d;
  wide.total_q = 1 << 20;
  wide.max_q_len = 1 << 14;
  EXPECT_ST(st(wide, 4096), SPA_ERR_UNSUPPORTED);
  EXPECT(stub::launches.empty());
  // no rows: mass and keep may be NULL
  spa_dims_t d0b = d;
  d0b.total_q = 0;
  EXPECT_ST(st(d0b, 2, 0.5, 0, I32, nullptr, nullptr), SPA_OK);
  reset();
  EXPECT_ST(st(d, 2, 1.0, 3), SPA_OK);
  EXPECT(launched({"select_tokens"}));
}

static void validate_paths() {
  spa_dims_t d = dims();
  Buf wsb(256);
  void* W = wsb.at();
  int32_t code = -7;
  int64_t index = -7;
  auto val = [&](void* ws, size_t n, const int32_t* ctx = I32, int64_t cap = 100) {
    return seg_paged_attn_validate(&d, ctx, I32, I32, I32, I32, I32, cap, &code, &index, ws, n,
                                   nullptr);
  };
  reset();
  EXPECT_ST(val(W, 64, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(val(W, 64, I32, -1), SPA_ERR_INVALID_ARG);
  EXPECT_ST(val(nullptr, 64), SPA_ERR_WORKSPACE);
  EXPECT_ST(val(W, 63), SPA_ERR_WORKSPACE);
  EXPECT(stub::launches.empty());
  EXPECT_ST(val(W, 64), SPA_OK);
  EXPECT(code == 0 && index == -1);
  EXPECT(launched({"validate"}));
  reset();
  stub::validate_reports_bad = true;
  EXPECT_ST(val(W, 64), SPA_ERR_BAD_DATA);
  EXPECT(code == 3 && index == 17);
  // bad_code and bad_index may be NULL
  EXPECT_ST(seg_paged_attn_validate(&d, I32, I32, I32, I32, I32, I32, 100, nullptr, nullptr, W, 64,
                                    nullptr), SPA_ERR_BAD_DATA);
  reset();
  stub::launch_result = hipErrorLaunchFailure;
  EXPECT_ST(val(W, 64), SPA_ERR_HIP);
}

static void status_and_profile_paths() {
  const int codes[] = {SPA_OK, SPA_ERR_INVALID_ARG, SPA_ERR_UNSUPPORTED, SPA_ERR_WORKSPACE,
                       SPA_ERR_CAPACITY, SPA_ERR_HIP, SPA_ERR_BAD_DATA};
  for (int c : codes) {
    const char* s = seg_paged_attn_status_string((spa_status_t)c);
    EXPECT(s != nullptr && std::strcmp(s, "unknown status") != 0);
  }
  EXPECT(std::strcmp(seg_paged_attn_status_string((spa_status_t)-99), "unknown status") == 0);
  EXPECT(std::strcmp(seg_paged_attn_status_string((spa_status_t)12345), "unknown status") == 0);

  // timing hooks: every launch between begin and end is counted per kind
  spa_dims_t d = dims();
  const size_t ws = seg_paged_attn_workspace_size(&d, SPA_SEL_ALL);
  Buf wsb(ws + 64);
  reset();
  EXPECT_ST(seg_paged_attn_profile_begin(), SPA_OK);
  for (int i = 0; i < 3; ++i)
    EXPECT_ST(seg_paged_attn_fwd(&d, A, I32, I32, A, A2, I32, I32, I32, I32, 1 << 20, A2, nullptr,
                                 wsb.at(), ws, nullptr), SPA_OK);
  EXPECT_ST(seg_paged_attn_page_summary(&d, A, I32, (float*)A2, nullptr), SPA_OK);
  const char* names[8] = {};
  int32_t counts[8] = {};
  double ms[8] = {};
  const int32_t n = seg_paged_attn_profile_end(names, counts, ms, 8);
  EXPECT(n == 3);
  if (n == 3) {
    EXPECT(std::strcmp(names[0], "decode_attn") == 0 && counts[0] == 3);
    EXPECT(std::strcmp(names[1], "combine") == 0 && counts[1] == 3);
    EXPECT(std::strcmp(names[2], "page_summary") == 0 && counts[2] == 1);
    EXPECT(std::fabs(ms[0] - 1.5) < 1e-9);
  }
  // a smaller cap fills only that many kinds but still counts them all
  EXPECT_ST(seg_paged_attn_profile_begin(), SPA_OK);
  EXPECT_ST(seg_paged_attn_page_summary(&d, A, I32, (float*)A2, nullptr), SPA_OK);
  EXPECT_ST(seg_paged_attn_rope_align(&d, A, I32, I32, 4, 1e4, nullptr), SPA_OK);
  const char* one[1] = {};
  EXPECT(seg_paged_attn_profile_end(one, nullptr, nullptr, 1) == 2);
  EXPECT(one[0] != nullptr && std::strcmp(one[0], "page_summary") == 0);
  // end without begin: nothing recorded
  EXPECT(seg_paged_attn_profile_end(nullptr, nullptr, nullptr, 0) == 0);
  // begin twice drops the earlier records (their events are released)
  EXPECT_ST(seg_paged_attn_profile_begin(), SPA_OK);
  EXPECT_ST(seg_paged_attn_page_summary(&d, A, I32, (float*)A2, nullptr), SPA_OK);
  EXPECT_ST(seg_paged_attn_profile_begin(), SPA_OK);
  EXPECT(seg_paged_attn_profile_end(nullptr, nullptr, nullptr, 0) == 0);
}

static void noalloc_paths() {
  // the first lookup of the built-in scratch fails: reported, nothing launched
  spa_dims_t d = dims();
  auto call = [&](const spa_dims_t& dd, const void* q = A, void* out = A2) {
    return seg_paged_attn_fwd_noalloc(&dd, q, I32, I32, A, A2, I32, I32, I32, I32, 1 << 20, out,
                                      (float*)A, nullptr);
  };
  reset();
  stub::symbol_lookup_fails = true;
  EXPECT_ST(call(d), SPA_ERR_HIP);
  EXPECT(stub::launches.empty());
  stub::symbol_lookup_fails = false;
  // then found once and kept for the device
  EXPECT_ST(call(d), SPA_OK);
  EXPECT(launched({"decode_attn", "combine"}));
  const float* first = stub::last_part_o;
  EXPECT(first != nullptr);
  const int lookups = stub::symbol_lookups;
  reset();
  EXPECT_ST(call(d), SPA_OK);
  EXPECT(stub::symbol_lookups == lookups);
  EXPECT(stub::last_part_o == first);
  // the same argument checks as seg_paged_attn_fwd
  EXPECT_ST(call(d, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(call(d, A, nullptr), SPA_ERR_INVALID_ARG);
  EXPECT_ST(call(d, MIS16), SPA_ERR_INVALID_ARG);
  spa_dims_t bad = d;
  bad.head_dim = 48;
  EXPECT_ST(call(bad), SPA_ERR_UNSUPPORTED);
  EXPECT_ST(seg_paged_attn_fwd_noalloc(nullptr, A, I32, I32, A, A2, I32, I32, I32, I32, 1 << 20, A2,
                                       nullptr, nullptr), SPA_ERR_INVALID_ARG);
  // partials beyond the scratch: refused before any launch
  reset();
  spa_dims_t big = dims(1024, 64, 8, 128, 16, 4, 4, 15, 1024 * 15);  // 8192 units x 8 row blocks
  EXPECT(seg_paged_attn_workspace_size(&big, SPA_SEL_ALL) > SPA_NOALLOC_SCRATCH_BYTES);
  EXPECT_ST(call(big), SPA_ERR_WORKSPACE);
  EXPECT(stub::launches.empty());
  // the largest decode shape that fits runs; chunked prefill keeps no partials
  spa_dims_t fit = dims(376, 32, 8, 128, 16, 4, 4, 1, 376);           // 3008 units x 1 row block
  EXPECT(seg_paged_attn_workspace_size(&fit, SPA_SEL_ALL) <= SPA_NOALLOC_SCRATCH_BYTES);
  EXPECT_ST(call(fit), SPA_OK);
  EXPECT(launched({"decode_attn", "combine"}));
  reset();
  spa_dims_t pre = dims(1024, 64, 8, 128, 16, 4, 4, 512, 1024 * 512);
  EXPECT_ST(call(pre), SPA_OK);
  EXPECT(launched({"prefill_attn"}));
}

static void validate_switch_paths() {
  spa_dims_t d = dims();
  const size_t ws = seg_paged_attn_workspace_size(&d, SPA_SEL_ALL);
  Buf wsb(ws + 64);
  auto fwd = [&]() {
    return seg_paged_attn_fwd(&d, A, I32, I32, A, A2, I32, I32, I32, I32, 1 << 20, A2, nullptr,
                              wsb.at(), ws, nullptr);
  };
  reset();
  setenv("SEGPA_VALIDATE", "1", 1);
  EXPECT_ST(fwd(), SPA_OK);                   // lists found valid: checked, then launched
  EXPECT(launched({"validate", "decode_attn", "combine"}));
  reset();
  stub::validate_reports_bad = true;
  EXPECT_ST(fwd(), SPA_ERR_BAD_DATA);         // bad lists: nothing launched after the check
  EXPECT(launched({"validate"}));
  reset();
  setenv("SEGPA_VALIDATE", "0", 1);
  stub::validate_reports_bad = true;
  EXPECT_ST(fwd(), SPA_OK);                   // switched off: no check
  EXPECT(launched({"decode_attn", "combine"}));
  unsetenv("SEGPA_VALIDATE");
  reset();
}

int main() {
  validate_switch_paths();
  noalloc_paths();
  check_dims_paths();
  select_paths();
  fwd_paths();
  summary_append_rope_paths();
  token_paths();
  validate_paths();
  status_and_profile_paths();
  std::printf("%d cases, %d failed\n", g_cases, g_fail);
  return g_fail == 0 ? 0 : 1;
}
