// Host runtime of libcofie: thread-local error strings, the per-dispatch kernel
// timer, the scratch arena and device queries.
#include <cstdarg>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

namespace cofie {

// ---- errors -------------------------------------------------------------------
static thread_local char g_err[512] = "";

int set_error(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

void clear_error() { g_err[0] = '\0'; }

// ---- kernel timing ------------------------------------------------------------
namespace {
struct Record {
  std::string name;
  hipEvent_t start, stop;
};
struct Profiler {
  std::mutex mu;
  bool on = false;
  std::vector<Record> recs;        // events recorded since the last reset
  std::vector<hipEvent_t> spare;   // events kept for reuse
  hipEvent_t get() {
    if (!spare.empty()) {
      hipEvent_t e = spare.back();
      spare.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};
Profiler& prof() {
  static Profiler* p = new Profiler();  // never destroyed: events outlive static teardown
  return *p;
}
}  // namespace

bool prof_slot(const char* name, hipEvent_t* start, hipEvent_t* stop) {
  Profiler& p = prof();
  std::lock_guard<std::mutex> lk(p.mu);
  if (!p.on) return false;
  hipEvent_t a = p.get(), b = p.get();
  if (!a || !b) {
    if (a) p.spare.push_back(a);
    if (b) p.spare.push_back(b);
    return false;
  }
  p.recs.push_back({name, a, b});
  *start = a;
  *stop = b;
  return true;
}

// ---- LDS attribute cache ----------------------------------------------------------
namespace {
std::mutex g_lds_mu;
std::map<const void*, size_t>& lds_sizes() {
  static auto* m = new std::map<const void*, size_t>();
  return *m;
}
}  // namespace

bool lds_attr_done(const void* kernel, size_t bytes) {
  std::lock_guard<std::mutex> lk(g_lds_mu);
  auto it = lds_sizes().find(kernel);
  return it != lds_sizes().end() && it->second >= bytes;
}

void lds_attr_mark(const void* kernel, size_t bytes) {
  std::lock_guard<std::mutex> lk(g_lds_mu);
  size_t& v = lds_sizes()[kernel];
  if (bytes > v) v = bytes;
}

// ---- scratch ------------------------------------------------------------------
static void raise_pool_threshold(hipStream_t) {
  static std::once_flag once;
  std::call_once(once, [] {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return;
    hipMemPool_t pool;
    if (hipDeviceGetDefaultMemPool(&pool, dev) != hipSuccess) return;
    uint64_t keep = ~uint64_t(0);  // keep freed blocks in the pool between calls
    (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
  });
}

int Scratch::acquire(void* ws, size_t ws_bytes, size_t need, hipStream_t s) {
  if (!ws && need > 0 && dry_run())
    return set_error(COFIE_EINVAL, "a dry run allocates nothing: pass a workspace of %zu bytes", need);
  if (ws) {
    if (ws_bytes < need)
      return set_error(COFIE_ENOMEM, "workspace of %zu bytes is smaller than the %zu required",
                       ws_bytes, need);
    base_ = static_cast<char*>(ws);
    return COFIE_OK;
  }
  if (need == 0) return COFIE_OK;
  raise_pool_threshold(s);
  void* p = nullptr;
  hipError_t e = hipMallocAsync(&p, need, s);
  if (e != hipSuccess || !p)
    return set_error(COFIE_ENOMEM, "hipMallocAsync(%zu) failed: %s", need, hipGetErrorString(e));
  base_ = static_cast<char*>(p);
  owned_ = true;
  stream_ = s;
  return COFIE_OK;
}

Scratch::~Scratch() {
  if (owned_ && base_) (void)hipFreeAsync(base_, stream_);
}

// ---- dry run ----------------------------------------------------------------------
namespace {
struct DryState {
  bool on = false;
  struct Buf {
    uintptr_t base;
    size_t bytes;
    std::string name;
  };
  std::vector<Buf> bufs;
  size_t hit = 0;  // the buffer of the last lookup
  std::map<uintptr_t, std::vector<uint8_t>> shadows;
  int64_t checked = 0, violations = 0;
  std::string first;
};
thread_local DryState g_dry;

void dry_violation(const char* what, const char* fmt, long long a, long long b, long long c) {
  ++g_dry.violations;
  if (g_dry.first.empty()) {
    char msg[512];
    snprintf(msg, sizeof msg, fmt, what, a, b, c);
    g_dry.first = msg;
  }
}
}  // namespace

bool dry_run() { return g_dry.on; }

void dry_access(const void* base, int64_t off, int64_t bytes, const char* what) {
  ++g_dry.checked;
  const uintptr_t b = reinterpret_cast<uintptr_t>(base);
  const size_t nb = g_dry.bufs.size();
  for (size_t i = 0; i < nb; ++i) {
    const size_t k = (g_dry.hit + i) % nb;
    const auto& buf = g_dry.bufs[k];
    if (b >= buf.base && b < buf.base + buf.bytes) {
      g_dry.hit = k;
      const int64_t lo = (int64_t)(b - buf.base) + off;
      if (lo < 0 || lo + bytes > (int64_t)buf.bytes)
        dry_violation(what, "%s: bytes [%lld, %lld) outside a buffer of %lld", (long long)lo, (long long)(lo + bytes),
                      (long long)buf.bytes);
      return;
    }
  }
  dry_violation(what, "%s: base %llx (+%lld, %lld bytes) in no registered buffer", (long long)b, (long long)off,
                (long long)bytes);
}

void dry_range(int64_t v, int64_t lo, int64_t hi, const char* what) {
  ++g_dry.checked;
  if (v < lo || v >= hi) dry_violation(what, "%s: %lld outside [%lld, %lld)", (long long)v, (long long)lo, (long long)hi);
}

int copy_to_device(void* dst, const void* src, size_t bytes, hipStream_t s, const char* what) {
  if (bytes == 0) return COFIE_OK;
  if (dry_run()) {
    dry_access(dst, 0, (int64_t)bytes, what);
    const auto* p = static_cast<const uint8_t*>(src);
    g_dry.shadows[reinterpret_cast<uintptr_t>(dst)] = std::vector<uint8_t>(p, p + bytes);
    return COFIE_OK;
  }
  if (hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, s) != hipSuccess)
    return set_error(COFIE_EHIP, "copying %s to the device failed", what);
  return COFIE_OK;
}

const void* dry_shadow(const void* dst) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(dst);
  auto it = g_dry.shadows.upper_bound(a);  // the first copy past a; the one before may hold it
  if (it == g_dry.shadows.begin()) return nullptr;
  --it;
  if (a >= it->first + it->second.size()) return nullptr;
  return it->second.data() + (a - it->first);
}

void dry_lds(int64_t off, int64_t bytes, int64_t lds_bytes, const char* what) {
  ++g_dry.checked;
  if (off < 0 || off + bytes > lds_bytes)
    dry_violation(what, "%s: LDS bytes [%lld, %lld) outside %lld", (long long)off, (long long)(off + bytes),
                  (long long)lds_bytes);
}

int device_cu_count() {
  static int cached[64] = {0};
  if (dry_run()) return 256;  // MI355X: the plans the address check walks are the GPU's
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
    cached[dev] = cus;
  }
  return cached[dev];
}

}  // namespace cofie

// ---- exported profiler / error API ------------------------------------------------
extern "C" {

const char* cofie_last_error(void) { return cofie::g_err; }

const char* cofie_version(void) { return "cofie-mi355x 0.1.0 (gfx950)"; }

int cofie_profiler_enable(int on) {
  auto& p = cofie::prof();
  std::lock_guard<std::mutex> lk(p.mu);
  p.on = on != 0;
  return COFIE_OK;
}

int cofie_profiler_reset(void) {
  auto& p = cofie::prof();
  std::lock_guard<std::mutex> lk(p.mu);
  for (auto& r : p.recs) {
    (void)hipEventSynchronize(r.stop);
    p.spare.push_back(r.start);
    p.spare.push_back(r.stop);
  }
  p.recs.clear();
  return COFIE_OK;
}

int cofie_profiler_read(const char* name_substr, double* total_ms, int64_t* launches) {
  if (!total_ms || !launches) return cofie::set_error(COFIE_EINVAL, "null output pointer");
  auto& p = cofie::prof();
  std::lock_guard<std::mutex> lk(p.mu);
  double sum = 0;
  int64_t cnt = 0;
  for (auto& r : p.recs) {
    if (name_substr && !strstr(r.name.c_str(), name_substr)) continue;
    if (hipEventSynchronize(r.stop) != hipSuccess)
      return cofie::set_error(COFIE_EHIP, "event synchronisation failed");
    float ms = 0;
    if (hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess)
      return cofie::set_error(COFIE_EHIP, "hipEventElapsedTime failed");
    sum += ms;
    ++cnt;
  }
  *total_ms = sum;
  *launches = cnt;
  return COFIE_OK;
}

int cofie_debug_dry_run(int on) {
  cofie::g_dry = cofie::DryState();
  cofie::g_dry.on = on != 0;
  return COFIE_OK;
}

int cofie_debug_buffer(const void* base, size_t bytes, const char* name) {
  if (!base) return cofie::set_error(COFIE_EINVAL, "buffer base is NULL");
  cofie::g_dry.bufs.push_back({reinterpret_cast<uintptr_t>(base), bytes, name ? name : "?"});
  return COFIE_OK;
}

int cofie_debug_buffer_data(const void* base, const void* data, size_t bytes, const char* name) {
  const int rc = cofie_debug_buffer(base, bytes, name);
  if (rc || !bytes) return rc;
  if (!data) return cofie::set_error(COFIE_EINVAL, "data is NULL");
  const auto* p = static_cast<const uint8_t*>(data);
  cofie::g_dry.shadows[reinterpret_cast<uintptr_t>(base)] = std::vector<uint8_t>(p, p + bytes);
  return COFIE_OK;
}

int64_t cofie_debug_dry_run_result(int64_t* checked, char* msg, size_t msg_bytes) {
  if (checked) *checked = cofie::g_dry.checked;
  if (msg && msg_bytes) snprintf(msg, msg_bytes, "%s", cofie::g_dry.first.c_str());
  return cofie::g_dry.violations;
}

}  // extern "C"
