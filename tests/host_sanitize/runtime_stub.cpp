// Host-only stand-ins for the HIP runtime calls and the kernel launchers that
// the library's host code (csrc/api.cpp) makes. Linked with api.cpp into a
// sanitized host program, they let every argument check, workspace rule and
// launch decision run under AddressSanitizer and UndefinedBehaviorSanitizer
// without a GPU. No kernel code is compiled into that program.
#include "runtime_stub.hpp"

#include <cstdlib>
#include <cstring>
#include <string>

namespace stub {
std::vector<std::string> launches;
hipError_t launch_result = hipSuccess;
bool validate_reports_bad = false;
int cus = 256;
bool symbol_lookup_fails = false;
int symbol_lookups = 0;
const float* last_part_o = nullptr;

// Reads every field a launcher hands to a kernel, so a value built from
// uninitialised or out-of-range host data is touched (and caught) here.
template <class T>
static void touch(const T& a) {
  volatile unsigned char sink = 0;
  const unsigned char* p = reinterpret_cast<const unsigned char*>(&a);
  for (size_t i = 0; i < sizeof(T); ++i) sink ^= p[i];
  (void)sink;
}

static hipError_t record(const char* name) {
  launches.emplace_back(name);
  return launch_result;
}
}  // namespace stub

// ---- HIP runtime ---------------------------------------------------------------
struct StubEvent {
  double t;
};

extern "C" {
hipError_t hipGetDevice(int* d) {
  if (d == nullptr) return hipErrorInvalidValue;
  *d = 0;
  return hipSuccess;
}
hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t attr, int) {
  if (v == nullptr) return hipErrorInvalidValue;
  *v = attr == hipDeviceAttributeMultiprocessorCount ? stub::cus : 1;
  return hipSuccess;
}
hipError_t hipEventCreate(hipEvent_t* e) {
  if (e == nullptr) return hipErrorInvalidValue;
  *e = reinterpret_cast<hipEvent_t>(new StubEvent{0.0});
  return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t e) {
  delete reinterpret_cast<StubEvent*>(e);
  return hipSuccess;
}
hipError_t hipEventSynchronize(hipEvent_t e) { return e ? hipSuccess : hipErrorInvalidHandle; }
hipError_t hipEventElapsedTime(float* ms, hipEvent_t a, hipEvent_t b) {
  if (ms == nullptr || a == nullptr || b == nullptr) return hipErrorInvalidValue;
  *ms = 0.5f;
  return hipSuccess;
}
hipError_t hipMemsetAsync(void* p, int v, size_t n, hipStream_t) {
  std::memset(p, v, n);
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t n, hipMemcpyKind, hipStream_t) {
  std::memcpy(dst, src, n);
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
// the scratch's "device address" is its host-side stand-in here (never dereferenced)
hipError_t hipGetSymbolAddress(void** p, const void* symbol) {
  ++stub::symbol_lookups;
  if (p == nullptr || symbol == nullptr) return hipErrorInvalidValue;
  if (stub::symbol_lookups == 1 && stub::symbol_lookup_fails) return hipErrorInvalidSymbol;
  *p = const_cast<void*>(symbol);
  return hipSuccess;
}

// code-object registration of the library's device variables (nothing to load here)
static void* g_module = nullptr;
void** __hipRegisterFatBinary(const void*) { return &g_module; }
void __hipUnregisterFatBinary(void**) {}
void __hipRegisterVar(void**, void*, char*, char*, int, size_t, int, int) {}
// the embedded code-object bundle the host code refers to (its name comes from
// the compilation unit id and is passed in by the build)
unsigned char SEGPA_FATBIN_SYMBOL[16] = {0};
}

// ---- kernel launchers ------------------------------------------------------------
namespace segpa {
hipError_t launch_decode(const FwdArgs& a, hipStream_t) {
  stub::touch(a);
  stub::last_part_o = a.part_o;
  return stub::record("decode_attn");
}
hipError_t launch_combine(const FwdArgs& a, hipStream_t) {
  stub::touch(a);
  return stub::record("combine");
}
hipError_t launch_prefill(const FwdArgs& a, hipStream_t) {
  stub::touch(a);
  return stub::record("prefill_attn");
}
hipError_t launch_rope_align(const RopeArgs& a, hipStream_t) {
  stub::touch(a);
  return stub::record("rope_align");
}
hipError_t launch_append(const AppendArgs& a, hipStream_t) {
  stub::touch(a);
  return stub::record("append");
}
hipError_t launch_select_scores(const SelArgs& a, hipStream_t) {
  stub::touch(a);
  return stub::record("select_score");
}
hipError_t launch_select_fill(const SelArgs& a, hipStream_t) {
  stub::touch(a);
  return stub::record("select_fill");
}
hipError_t launch_token_mass(const MassArgs& a, hipStream_t) {
  stub::touch(a);
  return stub::record("token_mass");
}
hipError_t launch_select_tokens(const TokSelArgs& a, hipStream_t) {
  stub::touch(a);
  return stub::record("select_tokens");
}
hipError_t launch_page_summary(const SummaryArgs& a, hipStream_t) {
  stub::touch(a);
  return stub::record("page_summary");
}
hipError_t launch_validate(const ValidateArgs& a, hipStream_t) {
  stub::touch(a);
  if (stub::validate_reports_bad) a.result[2] = 17;  // a bad selected page at index 17
  return stub::record("validate");
}
int decode_blocks_per_cu(int, int) { return 2; }
int prefill_rows_per_block() { return 256; }
int token_mass_keys_per_block() { return 512; }
}  // namespace segpa
