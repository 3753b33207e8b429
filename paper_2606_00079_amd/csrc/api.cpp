// Host side of libbitsmoe: errors, scratch memory, the LAPACK-backed shared
// basis (step 2) and the packed layout.
#include <dlfcn.h>
#include <hip/hip_runtime_api.h>

#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "bitsmoe.h"
#include "internal.hpp"

namespace bitsmoe {

static thread_local std::string g_last_error;

bitsmoe_status fail(bitsmoe_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

bitsmoe_status ok() {
  g_last_error.clear();
  return BITSMOE_OK;
}

bitsmoe_status device_error(const char* what, int hip_err) {
  char buf[256];
  std::snprintf(buf, sizeof buf, "%s: HIP error %d (%s)", what, hip_err,
                hipGetErrorString(static_cast<hipError_t>(hip_err)));
  return fail(BITSMOE_ERR_DEVICE, buf);
}

int device_cus() {
  static std::mutex mu;
  static std::map<int, int> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return 256;
  }
  std::lock_guard<std::mutex> lock(mu);
  auto it = cache.find(dev);
  if (it != cache.end()) return it->second;
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) {
    (void)hipGetLastError();
    n = 256;
  }
  cache[dev] = n;
  return n;
}

// ----------------------------------------------------------------------------
// scratch
// ----------------------------------------------------------------------------
namespace {
struct DeviceScratch {
  void* ptr[kScratchCount] = {};
  size_t size[kScratchCount] = {};
};
std::mutex g_scratch_mu;
std::map<int, DeviceScratch> g_scratch;
}  // namespace

void* scratch(int slot, size_t bytes, void* stream, bitsmoe_status* st) {
  *st = BITSMOE_OK;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    *st = device_error("hipGetDevice", e);
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  DeviceScratch& ds = g_scratch[dev];
  if (bytes == 0) bytes = 256;
  if (ds.size[slot] >= bytes) return ds.ptr[slot];
  // Round up to 2 MiB so that a sequence of slightly growing calls does not
  // reallocate every time.
  size_t want = (bytes + (size_t(2) << 20) - 1) & ~((size_t(2) << 20) - 1);
  if (ds.ptr[slot]) {
    e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
      *st = device_error("hipStreamSynchronize (scratch growth)", e);
      return nullptr;
    }
    (void)hipFree(ds.ptr[slot]);
    ds.ptr[slot] = nullptr;
    ds.size[slot] = 0;
  }
  void* p = nullptr;
  e = hipMalloc(&p, want);
  if (e != hipSuccess || p == nullptr) {
    (void)hipGetLastError();
    char buf[160];
    std::snprintf(buf, sizeof buf, "scratch: cannot allocate %zu bytes on device %d", want, dev);
    *st = fail(BITSMOE_ERR_NOMEM, buf);
    return nullptr;
  }
  ds.ptr[slot] = p;
  ds.size[slot] = want;
  return p;
}

// ----------------------------------------------------------------------------
// kernel timing
// ----------------------------------------------------------------------------
namespace {
struct TimedLaunch {
  std::string name;
  hipEvent_t start, stop;
};
std::mutex g_timing_mu;
bool g_timing = false;
std::string g_timing_only;  // empty: every timed launch
std::vector<TimedLaunch> g_launches;
// Events read back by bitsmoe_kernel_time are kept for reuse, per device:
// creating an event costs the host more than recording one, and between two
// short kernels that cost shows up on the device as idle time.
std::map<int, std::vector<hipEvent_t>> g_event_pool;

// (with g_timing_mu held)
hipError_t take_event(hipEvent_t* e) {
  int dev = 0;
  hipError_t st = hipGetDevice(&dev);
  if (st != hipSuccess) return st;
  std::vector<hipEvent_t>& pool = g_event_pool[dev];
  if (!pool.empty()) {
    *e = pool.back();
    pool.pop_back();
    return hipSuccess;
  }
  return hipEventCreate(e);
}
void give_event(hipEvent_t e) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipEventDestroy(e);
    return;
  }
  g_event_pool[dev].push_back(e);
}
}  // namespace

KernelTimer::KernelTimer(const char* name, void* stream) : name_(name), stream_(stream) {
  if (!name) return;  // an untimed launch: no events
  std::lock_guard<std::mutex> lock(g_timing_mu);
  if (!g_timing || (!g_timing_only.empty() && g_timing_only != name)) return;
  hipEvent_t e;
  if (take_event(&e) != hipSuccess) return;
  if (hipEventRecord(e, static_cast<hipStream_t>(stream)) != hipSuccess) {
    (void)hipEventDestroy(e);
    return;
  }
  start_ = e;
}

KernelTimer::~KernelTimer() {
  if (!start_) return;
  std::lock_guard<std::mutex> lock(g_timing_mu);
  hipEvent_t e;
  if (take_event(&e) != hipSuccess) {
    (void)hipEventDestroy(static_cast<hipEvent_t>(start_));
    return;
  }
  if (hipEventRecord(e, static_cast<hipStream_t>(stream_)) != hipSuccess) {
    (void)hipEventDestroy(e);
    (void)hipEventDestroy(static_cast<hipEvent_t>(start_));
    return;
  }
  g_launches.push_back({name_, static_cast<hipEvent_t>(start_), e});
}

// ----------------------------------------------------------------------------
// LAPACK (dsyevd) loaded at run time
// ----------------------------------------------------------------------------
namespace {
typedef void (*dsyevd32_t)(const char*, const char*, const int32_t*, double*, const int32_t*,
                           double*, double*, const int32_t*, int32_t*, const int32_t*, int32_t*,
                           size_t, size_t);
typedef void (*dsyevd64_t)(const char*, const char*, const int64_t*, double*, const int64_t*,
                           double*, double*, const int64_t*, int64_t*, const int64_t*, int64_t*,
                           size_t, size_t);
struct Lapack {
  void* handle = nullptr;
  dsyevd32_t f32 = nullptr;
  dsyevd64_t f64 = nullptr;
  std::string path;
};
std::mutex g_lapack_mu;
Lapack g_lapack;
std::string g_lapack_path;  // set by bitsmoe_set_lapack

bool load_lapack_locked(std::string* why) {
  if (g_lapack.handle) return true;
  std::vector<std::string> cands;
  if (!g_lapack_path.empty()) cands.push_back(g_lapack_path);
  if (const char* env = std::getenv("BITSMOE_LAPACK")) cands.push_back(env);
  cands.push_back("liblapack.so.3");
  cands.push_back("liblapack.so");
  std::string tried;
  for (const std::string& c : cands) {
    void* h = dlopen(c.c_str(), RTLD_NOW | RTLD_LOCAL);
    if (!h) {
      tried += " " + c + " (not loadable)";
      continue;
    }
    // ILP64 names first: their integer width is unambiguous.
    const char* n64[] = {"scipy_dsyevd_64_", "dsyevd_64_", "dsyevd64_"};
    for (const char* n : n64) {
      if (void* s = dlsym(h, n)) {
        g_lapack.handle = h;
        g_lapack.f64 = reinterpret_cast<dsyevd64_t>(s);
        g_lapack.path = c;
        return true;
      }
    }
    if (void* s = dlsym(h, "dsyevd_")) {
      g_lapack.handle = h;
      g_lapack.f32 = reinterpret_cast<dsyevd32_t>(s);
      g_lapack.path = c;
      return true;
    }
    tried += " " + c + " (no dsyevd)";
    dlclose(h);
  }
  *why = "no LAPACK with dsyevd found; tried:" + tried +
         " (set one with bitsmoe_set_lapack or BITSMOE_LAPACK)";
  return false;
}

// Full eigendecomposition of the symmetric n x n matrix A (overwritten by the
// eigenvectors, eigenvector k contiguous at A + k*n); w ascending.
bitsmoe_status eig_sym(double* A, int64_t n, double* w) {
  std::lock_guard<std::mutex> lock(g_lapack_mu);
  std::string why;
  if (!load_lapack_locked(&why)) return fail(BITSMOE_ERR_UNAVAILABLE, why);
  const char jobz = 'V', uplo = 'U';
  if (g_lapack.f64) {
    int64_t N = n, lda = n, lwork = -1, liwork = -1, info = 0, iq = 0;
    double wq = 0;
    g_lapack.f64(&jobz, &uplo, &N, A, &lda, w, &wq, &lwork, &iq, &liwork, &info, 1, 1);
    if (info != 0) return fail(BITSMOE_ERR_NUMERIC, "dsyevd workspace query failed");
    lwork = static_cast<int64_t>(wq) + 1;
    liwork = iq;
    std::vector<double> work(static_cast<size_t>(lwork));
    std::vector<int64_t> iwork(static_cast<size_t>(liwork));
    g_lapack.f64(&jobz, &uplo, &N, A, &lda, w, work.data(), &lwork, iwork.data(), &liwork, &info,
                 1, 1);
    if (info != 0) return fail(BITSMOE_ERR_NUMERIC, "dsyevd failed (info=" + std::to_string(info) + ")");
    return BITSMOE_OK;
  }
  if (n > INT32_MAX) return fail(BITSMOE_ERR_SHAPE, "matrix too large for an LP64 LAPACK");
  int32_t N = static_cast<int32_t>(n), lda = N, lwork = -1, liwork = -1, info = 0, iq = 0;
  double wq = 0;
  g_lapack.f32(&jobz, &uplo, &N, A, &lda, w, &wq, &lwork, &iq, &liwork, &info, 1, 1);
  if (info != 0) return fail(BITSMOE_ERR_NUMERIC, "dsyevd workspace query failed");
  lwork = static_cast<int32_t>(wq) + 1;
  liwork = iq;
  std::vector<double> work(static_cast<size_t>(lwork));
  std::vector<int32_t> iwork(static_cast<size_t>(liwork));
  g_lapack.f32(&jobz, &uplo, &N, A, &lda, w, work.data(), &lwork, iwork.data(), &liwork, &info, 1,
               1);
  if (info != 0) return fail(BITSMOE_ERR_NUMERIC, "dsyevd failed (info=" + std::to_string(info) + ")");
  return BITSMOE_OK;
}

}  // namespace

}  // namespace bitsmoe

using namespace bitsmoe;

extern "C" {

const char* bitsmoe_last_error(void) { return g_last_error.c_str(); }

bitsmoe_status bitsmoe_timing(int enable) {
  std::lock_guard<std::mutex> lock(g_timing_mu);
  g_timing = enable != 0;
  return ok();
}

bitsmoe_status bitsmoe_timing_only(const char* name) {
  std::lock_guard<std::mutex> lock(g_timing_mu);
  g_timing_only = name ? name : "";
  return ok();
}

bitsmoe_status bitsmoe_kernel_time(const char* name, double* total_ms, int64_t* launches) {
  if (!name || !total_ms) return fail(BITSMOE_ERR_ARG, "kernel_time: null pointer");
  std::lock_guard<std::mutex> lock(g_timing_mu);
  double sum = 0.0;
  int64_t count = 0;
  std::vector<TimedLaunch> keep;
  bitsmoe_status st = BITSMOE_OK;
  for (TimedLaunch& t : g_launches) {
    if (t.name != name) {
      keep.push_back(t);
      continue;
    }
    float ms = 0.0f;
    hipError_t e = hipEventSynchronize(t.stop);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, t.start, t.stop);
    if (e != hipSuccess && st == BITSMOE_OK) st = device_error("kernel_time", e);
    sum += ms;
    ++count;
    give_event(t.start);
    give_event(t.stop);
  }
  g_launches.swap(keep);
  *total_ms = sum;
  if (launches) *launches = count;
  return st == BITSMOE_OK ? ok() : st;
}

const char* bitsmoe_version(void) { return "bitsmoe-mi355x 0.1 (gfx950)"; }

void bitsmoe_release(void) {
  {
    std::lock_guard<std::mutex> lock(g_timing_mu);
    for (auto& kv : g_event_pool)
      for (hipEvent_t e : kv.second) (void)hipEventDestroy(e);
    g_event_pool.clear();
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  int cur = 0;
  (void)hipGetDevice(&cur);
  for (auto& kv : g_scratch) {
    if (hipSetDevice(kv.first) != hipSuccess) continue;
    (void)hipDeviceSynchronize();
    for (int s = 0; s < kScratchCount; ++s) {
      if (kv.second.ptr[s]) (void)hipFree(kv.second.ptr[s]);
      kv.second.ptr[s] = nullptr;
      kv.second.size[s] = 0;
    }
  }
  (void)hipSetDevice(cur);
}

bitsmoe_status bitsmoe_set_lapack(const char* path) {
  if (!path || !*path) return fail(BITSMOE_ERR_ARG, "bitsmoe_set_lapack: empty path");
  std::lock_guard<std::mutex> lock(g_lapack_mu);
  if (g_lapack.handle && g_lapack.path == path) return ok();
  void* h = dlopen(path, RTLD_NOW | RTLD_LOCAL);
  if (!h) return fail(BITSMOE_ERR_UNAVAILABLE, std::string("cannot load ") + path);
  dlclose(h);
  g_lapack_path = path;
  if (g_lapack.handle) {  // switch on next use
    g_lapack = Lapack();
  }
  return ok();
}

bitsmoe_status bitsmoe_shared_basis(const double* M_dev, int64_t d_out, int64_t r, float* Ut_dev,
                                    double* eigvals_host, double* host_ms, void* stream) {
  auto t0 = std::chrono::steady_clock::now();
  if (!M_dev || !Ut_dev) return fail(BITSMOE_ERR_ARG, "shared_basis: null pointer");
  if (!aligned16({M_dev, Ut_dev}))
    return fail(BITSMOE_ERR_ARG, "shared_basis: device pointers must be 16-byte aligned");
  if (d_out <= 0 || r <= 0) return fail(BITSMOE_ERR_ARG, "shared_basis: non-positive size");
  if (r > d_out) return fail(BITSMOE_ERR_SHAPE, "shared_basis: r > d_out");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t nn = static_cast<size_t>(d_out) * static_cast<size_t>(d_out);
  std::vector<double> A;
  std::vector<double> w;
  std::vector<float> Ut;
  try {
    A.resize(nn);
    w.resize(static_cast<size_t>(d_out));
    Ut.resize(static_cast<size_t>(r) * static_cast<size_t>(d_out));
  } catch (...) {
    return fail(BITSMOE_ERR_NOMEM, "shared_basis: host allocation failed");
  }
  hipError_t e = hipMemcpyAsync(A.data(), M_dev, nn * sizeof(double), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return device_error("shared_basis: copy of M", e);
  for (size_t i = 0; i < nn; ++i)
    if (!std::isfinite(A[i])) return fail(BITSMOE_ERR_NUMERIC, "shared_basis: M is not finite");
  bitsmoe_status st = eig_sym(A.data(), d_out, w.data());
  if (st != BITSMOE_OK) return st;
  for (int64_t k = 0; k < r; ++k) {
    const int64_t src = d_out - 1 - k;  // eigenvalues ascend
    const double* v = A.data() + static_cast<size_t>(src) * d_out;
    int64_t imax = 0;
    double amax = -1.0;
    for (int64_t i = 0; i < d_out; ++i) {
      double a = std::fabs(v[i]);
      if (a > amax) {
        amax = a;
        imax = i;
      }
    }
    const double sg = v[imax] < 0 ? -1.0 : 1.0;
    float* dst = Ut.data() + static_cast<size_t>(k) * d_out;
    for (int64_t i = 0; i < d_out; ++i) dst[i] = static_cast<float>(sg * v[i]);
    if (eigvals_host) eigvals_host[k] = w[static_cast<size_t>(src)];
  }
  e = hipMemcpyAsync(Ut_dev, Ut.data(), Ut.size() * sizeof(float), hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return device_error("shared_basis: copy of U", e);
  if (host_ms) {
    auto t1 = std::chrono::steady_clock::now();
    *host_ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
  }
  return ok();
}

bitsmoe_status bitsmoe_pack_layout(const uint8_t* bits_host, int64_t units, int64_t d,
                                   int64_t* word_offsets_host) {
  if (!bits_host || !word_offsets_host) return fail(BITSMOE_ERR_ARG, "pack_layout: null pointer");
  if (units <= 0 || d <= 0) return fail(BITSMOE_ERR_ARG, "pack_layout: non-positive size");
  if (d % 64 != 0) return fail(BITSMOE_ERR_SHAPE, "pack_layout: d must be a multiple of 64");
  const int64_t wpp = d / 64;
  int64_t off = 0;
  word_offsets_host[0] = 0;
  for (int64_t u = 0; u < units; ++u) {
    const int b = bits_host[u];
    if (!(b == 0 || b == 16 || (b >= 1 && b <= BITSMOE_MAX_BITS)))
      return fail(BITSMOE_ERR_ARG, "pack_layout: width other than 0, 1..8, 16 at unit " + std::to_string(u));
    off += b * wpp;
    word_offsets_host[u + 1] = off;
  }
  return ok();
}

}  // extern "C"
