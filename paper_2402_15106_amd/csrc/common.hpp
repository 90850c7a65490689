// Internal helpers shared by the HIP sources of libdsmpnn (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>
#include <string>
#include <vector>
#include <algorithm>
#include <cstdio>
#include <cstdarg>

#include "../../include/dsmpnn.h"

struct dsmp_handle {
  int device = 0;
  hipStream_t stream = nullptr;
  int edge_algo = 0;   // DSMP_EDGE_AUTO / PER_EDGE / AGGREGATE
  int n_cu = 256;      // compute units of the device (sizes persistent grids)
  void* sample_scratch = nullptr;   // device address of the allocation-free sampling scratch
  std::string err;
  // kernel timing (opt-in)
  struct Mark {
    int cls;
    hipEvent_t a, b;
  };
  bool prof = false;
  std::vector<Mark> pending;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> pool;
  double tot_ms[DSMP_K_COUNT] = {};
  int64_t launches[DSMP_K_COUNT] = {};
};

namespace dsmp {

// Brackets the launches issued in its scope with a pair of events when the
// handle's timing is on.
struct ProfScope {
  dsmp_handle* h;
  int idx = -1;
  ProfScope(dsmp_handle* hh, int cls) : h(hh) {
    if (!h || !h->prof) return;
    std::pair<hipEvent_t, hipEvent_t> ev;
    if (!h->pool.empty()) {
      ev = h->pool.back();
      h->pool.pop_back();
    } else if (hipEventCreate(&ev.first) != hipSuccess || hipEventCreate(&ev.second) != hipSuccess) {
      return;
    }
    if (hipEventRecord(ev.first, h->stream) != hipSuccess) {
      h->pool.push_back(ev);
      return;
    }
    h->pending.push_back({cls, ev.first, ev.second});
    idx = (int)h->pending.size() - 1;
  }
  void end() {
    if (idx >= 0) (void)hipEventRecord(h->pending[idx].b, h->stream);
    idx = -1;
  }
  ~ProfScope() { end(); }
};

inline dsmp_status fail(dsmp_handle* h, dsmp_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  if (h) h->err = buf;
  return st;
}

#define DSMP_HIP(h, call)                                                              \
  do {                                                                                 \
    hipError_t e_ = (call);                                                            \
    if (e_ != hipSuccess)                                                              \
      return ::dsmp::fail((h), DSMP_HIP_ERROR, "%s failed: %s", #call,                 \
                          hipGetErrorString(e_));                                      \
  } while (0)

#define DSMP_LAUNCHED(h, what)                                                         \
  do {                                                                                 \
    hipError_t e_ = hipGetLastError();                                                 \
    if (e_ != hipSuccess)                                                              \
      return ::dsmp::fail((h), DSMP_HIP_ERROR, "launch of %s failed: %s", (what),      \
                          hipGetErrorString(e_));                                      \
  } while (0)

#define DSMP_CHECK(h, cond, st, ...)                                                   \
  do {                                                                                 \
    if (!(cond)) return ::dsmp::fail((h), (st), __VA_ARGS__);                          \
  } while (0)

// Bump allocator over a caller workspace; every sub-buffer is 256-byte aligned.
struct Carve {
  uintptr_t base;
  size_t off = 0;
  explicit Carve(void* p) : base(reinterpret_cast<uintptr_t>(p)) {}
  template <typename T>
  T* take(size_t count) {
    off = (off + 255) & ~size_t(255);
    T* p = reinterpret_cast<T*>(base + off);
    off += count * sizeof(T);
    return p;
  }
  size_t used() const { return (off + 255) & ~size_t(255); }
};

inline unsigned ceil_div(int64_t a, int64_t b) { return (unsigned)((a + b - 1) / b); }

// Device-wide exclusive scan of n uint32 counts into out[0..n] (out[n] = total),
// in three launches: per-block sums, a single-block scan of the sums, and the
// per-block scan with offsets.  tmp needs scan_tmp_elems(n) uint32.
constexpr int SCAN_BLOCK = 1024;
inline size_t scan_tmp_elems(int64_t n) { return (size_t)ceil_div(n, SCAN_BLOCK) + 1; }
dsmp_status exclusive_scan_u32(dsmp_handle* h, const uint32_t* in, int32_t* out, int64_t n,
                               uint32_t* tmp);

// Fill n uint32 words with a value (a kernel, not a memset node).
// p[0..n) = v, and q[0..n) = v in the same launch when q is given
dsmp_status fill_u32(dsmp_handle* h, uint32_t* p, int64_t n, uint32_t v, uint32_t* q = nullptr);

// SplitMix64 output number c+1 after seeding the state with `seed`
// (Steele, Lea, Flood, OOPSLA 2014; Stafford's Mix13 finaliser).
__device__ __forceinline__ uint64_t splitmix64(uint64_t seed, uint64_t c) {
  uint64_t z = seed + (c + 1ull) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

}  // namespace dsmp
