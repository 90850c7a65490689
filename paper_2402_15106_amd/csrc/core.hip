// Handle management, scan and fill utilities, node sampling and row gather.
#include "common.hpp"

#include <map>
#include <mutex>
#include <new>

using namespace dsmp;

// ------------------------------------------------------------------ scan

namespace {

__device__ __forceinline__ uint32_t block_exclusive_scan_1024(uint32_t v, uint32_t* sh,
                                                             uint32_t* total) {
  // 1024 threads = 16 waves; wave scans by shuffles, then a scan of wave sums.
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    uint32_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[wid] = x;
  __syncthreads();
  if (wid == 0) {
    uint32_t s = lane < 16 ? sh[lane] : 0u;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      uint32_t y = __shfl_up(s, o, 64);
      if (lane >= o) s += y;
    }
    if (lane < 16) sh[16 + lane] = s;
  }
  __syncthreads();
  uint32_t wave_off = wid > 0 ? sh[16 + wid - 1] : 0u;
  *total = sh[31];
  uint32_t r = wave_off + x - v;
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(1024) void k_scan_blocksums(const uint32_t* __restrict__ in,
                                                         int64_t n, uint32_t* __restrict__ sums) {
  __shared__ uint32_t sh[32];
  int64_t i = (int64_t)blockIdx.x * SCAN_BLOCK + threadIdx.x;
  uint32_t v = i < n ? in[i] : 0u;
  uint32_t tot;
  block_exclusive_scan_1024(v, sh, &tot);
  if (threadIdx.x == 0) sums[blockIdx.x] = tot;
}

__global__ __launch_bounds__(1024) void k_scan_sums(uint32_t* __restrict__ sums, int nb) {
  // exclusive scan of nb block sums in place, in chunks of 1024; sums[nb] = total
  __shared__ uint32_t sh[32];
  uint32_t carry = 0;
  for (int base = 0; base < nb; base += SCAN_BLOCK) {
    int i = base + threadIdx.x;
    uint32_t v = i < nb ? sums[i] : 0u;
    uint32_t tot;
    uint32_t ex = block_exclusive_scan_1024(v, sh, &tot);
    if (i < nb) sums[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) sums[nb] = carry;
}

__global__ __launch_bounds__(1024) void k_scan_final(const uint32_t* __restrict__ in, int64_t n,
                                                     const uint32_t* __restrict__ sums,
                                                     int32_t* __restrict__ out, int nb) {
  __shared__ uint32_t sh[32];
  int64_t i = (int64_t)blockIdx.x * SCAN_BLOCK + threadIdx.x;
  uint32_t v = i < n ? in[i] : 0u;
  uint32_t tot;
  uint32_t ex = block_exclusive_scan_1024(v, sh, &tot);
  if (i < n) out[i] = (int32_t)(sums[blockIdx.x] + ex);
  if (blockIdx.x == 0 && threadIdx.x == 0) out[n] = (int32_t)sums[nb];
}

// Exclusive scan of up to 16 * 1024 values by one workgroup in one launch:
// thread t takes SCAN_PER consecutive values, the per-thread totals are
// scanned across the block, and each thread writes its values' prefixes;
// out[n] = total.
constexpr int SCAN_PER = 16;
__global__ __launch_bounds__(1024) void k_scan_single(const uint32_t* __restrict__ in, int64_t n,
                                                      int32_t* __restrict__ out) {
  __shared__ uint32_t sh[32];
  const int64_t b = (int64_t)threadIdx.x * SCAN_PER;
  uint32_t v[SCAN_PER], sum = 0;
#pragma unroll
  for (int k = 0; k < SCAN_PER; ++k) {
    v[k] = b + k < n ? in[b + k] : 0u;
    sum += v[k];
  }
  uint32_t tot;
  uint32_t run = block_exclusive_scan_1024(sum, sh, &tot);
#pragma unroll
  for (int k = 0; k < SCAN_PER; ++k) {
    if (b + k < n) out[b + k] = (int32_t)run;
    run += v[k];
  }
  if (threadIdx.x == 0) out[n] = (int32_t)tot;
}

// p[0..n) = v, and q[0..n) = v too when q is not null (two arrays, one launch)
__global__ void k_fill_u32(uint32_t* p, uint32_t* q, int64_t n, uint32_t v) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) {
    p[i] = v;
    if (q) q[i] = v;
  }
}

}  // namespace

namespace dsmp {

dsmp_status exclusive_scan_u32(dsmp_handle* h, const uint32_t* in, int32_t* out, int64_t n,
                               uint32_t* tmp) {
  int nb = (int)ceil_div(n, SCAN_BLOCK);
  if (n <= (int64_t)SCAN_PER * 1024) {   // one launch
    hipLaunchKernelGGL(k_scan_single, dim3(1), dim3(1024), 0, h->stream, in, n, out);
    DSMP_LAUNCHED(h, "scan");
    return DSMP_OK;
  }
  if (nb == 0) {
    hipLaunchKernelGGL(k_scan_sums, dim3(1), dim3(1024), 0, h->stream, tmp, 0);
    hipLaunchKernelGGL(k_scan_final, dim3(1), dim3(1024), 0, h->stream, in, (int64_t)0, tmp, out, 0);
    DSMP_LAUNCHED(h, "scan");
    return DSMP_OK;
  }
  hipLaunchKernelGGL(k_scan_blocksums, dim3(nb), dim3(1024), 0, h->stream, in, n, tmp);
  hipLaunchKernelGGL(k_scan_sums, dim3(1), dim3(1024), 0, h->stream, tmp, nb);
  hipLaunchKernelGGL(k_scan_final, dim3(nb), dim3(1024), 0, h->stream, in, n, tmp, out, nb);
  DSMP_LAUNCHED(h, "scan");
  return DSMP_OK;
}

dsmp_status fill_u32(dsmp_handle* h, uint32_t* p, int64_t n, uint32_t v, uint32_t* q) {
  if (n <= 0) return DSMP_OK;
  unsigned g = ceil_div(n, 256);
  if (g > 4096) g = 4096;
  hipLaunchKernelGGL(k_fill_u32, dim3(g), dim3(256), 0, h->stream, p, q, n, v);
  DSMP_LAUNCHED(h, "fill");
  return DSMP_OK;
}

}  // namespace dsmp

// ------------------------------------------------------------------ handle

extern "C" int dsmp_version(void) { return 10000; }

// device address of the sampling scratch array on the current device (set-up
// of the allocation-free sampling entry point; defined with the array below)
static dsmp_status sample_scratch_setup(dsmp_handle* h);

extern "C" dsmp_status dsmp_create(dsmp_handle** out, int device) {
  if (!out) return DSMP_INVALID_ARG;
  *out = nullptr;
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || device < 0 || device >= n) return DSMP_INVALID_ARG;
  if (hipSetDevice(device) != hipSuccess) return DSMP_HIP_ERROR;
  dsmp_handle* h = new (std::nothrow) dsmp_handle();
  if (!h) return DSMP_HIP_ERROR;
  h->device = device;
  int cu = 0;
  if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, device) == hipSuccess && cu > 0) h->n_cu = cu;
  const dsmp_status st = sample_scratch_setup(h);
  if (st != DSMP_OK) {
    delete h;
    return st;
  }
  *out = h;
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_destroy(dsmp_handle* h) {
  if (!h) return DSMP_OK;
  for (auto& m : h->pending) { (void)hipEventDestroy(m.a); (void)hipEventDestroy(m.b); }
  for (auto& e : h->pool) { (void)hipEventDestroy(e.first); (void)hipEventDestroy(e.second); }
  delete h;
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_profile_enable(dsmp_handle* h, int enable) {
  if (!h) return DSMP_INVALID_ARG;
  h->prof = enable != 0;
  return DSMP_OK;
}

static dsmp_status drain_marks(dsmp_handle* h) {
  for (auto& m : h->pending) {
    DSMP_HIP(h, hipEventSynchronize(m.b));
    float ms = 0.0f;
    DSMP_HIP(h, hipEventElapsedTime(&ms, m.a, m.b));
    h->tot_ms[m.cls] += ms;
    h->launches[m.cls] += 1;
    h->pool.push_back({m.a, m.b});
  }
  h->pending.clear();
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_profile_reset(dsmp_handle* h) {
  if (!h) return DSMP_INVALID_ARG;
  dsmp_status st = drain_marks(h);
  for (int k = 0; k < DSMP_K_COUNT; ++k) { h->tot_ms[k] = 0.0; h->launches[k] = 0; }
  return st;
}

extern "C" dsmp_status dsmp_profile_read(dsmp_handle* h, int cls, double* total_ms, int64_t* launches) {
  if (!h) return DSMP_INVALID_ARG;
  DSMP_CHECK(h, cls >= 0 && cls < DSMP_K_COUNT && total_ms && launches, DSMP_INVALID_ARG,
             "bad profile query");
  dsmp_status st = drain_marks(h);
  if (st != DSMP_OK) return st;
  *total_ms = h->tot_ms[cls];
  *launches = h->launches[cls];
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_set_stream(dsmp_handle* h, void* stream) {
  if (!h) return DSMP_INVALID_ARG;
  h->stream = reinterpret_cast<hipStream_t>(stream);
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_set_edge_algorithm(dsmp_handle* h, int32_t algorithm) {
  if (!h) return DSMP_INVALID_ARG;
  DSMP_CHECK(h, algorithm == DSMP_EDGE_AUTO || algorithm == DSMP_EDGE_PER_EDGE || algorithm == DSMP_EDGE_AGGREGATE,
             DSMP_INVALID_ARG, "unknown edge algorithm %d", algorithm);
  h->edge_algo = algorithm;
  return DSMP_OK;
}

extern "C" const char* dsmp_last_error(const dsmp_handle* h) { return h ? h->err.c_str() : ""; }

// ------------------------------------------------------------------ sampling
//
// Selection of the s smallest SplitMix64 keys out of M by a 4-pass MSB-first
// radix select over 16-bit digits (the keys are recomputed every pass), then a
// stable compaction of the candidates whose key is <= the s-th smallest.  The
// keys are distinct (the mix is a bijection of the counter), so exactly s are
// kept.

namespace {

struct SelState {
  unsigned long long prefix;   // digits fixed so far
  unsigned long long rank;     // 1-based rank of the wanted key among the unfixed ones
};

constexpr int SAMPLE_CHUNK = 1024;   // candidates per block in the compaction
constexpr int SEL_BINS = 65536;      // 16-bit digits

// Histogram of digit (k >> shift) & 0xFFFF over the keys that match the fixed prefix.
__global__ __launch_bounds__(256) void k_sel_hist(int64_t M, uint64_t seed, const SelState* st, int shift,
                                                  uint32_t* __restrict__ hist) {
  const uint64_t prefix = st->prefix;
  const uint64_t himask = shift >= 48 ? 0ull : (~0ull << (shift + 16));
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < M; i += stride) {
    const uint64_t k = splitmix64(seed, (uint64_t)i);
    if ((k & himask) == (prefix & himask)) atomicAdd(&hist[(k >> shift) & 0xFFFFu], 1u);
  }
}

__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// One workgroup of 16 waves.  The histogram is read once, in 1 KB pieces
// that one wave loads whole: piece P = 16 w + v covers bins
// [256 P, 256 P + 256), lane l of it bins 256 P + 4 l .. + 3.  Every piece's
// total goes to LDS; wave 0 scans the 256 totals and finds the piece that
// holds the wanted rank; the wave that read that piece scans its lanes and
// fixes the digit.  Every wave clears the bins it read for the next pass.
__global__ __launch_bounds__(1024) void k_sel_pick(SelState* st, int shift, uint32_t* __restrict__ hist) {
  static_assert(SEL_BINS == 16 * 16 * 256, "16 waves x 16 pieces of 256 bins");
  __shared__ uint32_t psum[256];
  __shared__ uint32_t pick[2];   // the piece, and the count of the bins before it
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (threadIdx.x == 0) pick[0] = ~0u;
  uint4* hb = reinterpret_cast<uint4*>(hist) + (size_t)w * 1024 + lane;
  uint4 x[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) x[v] = hb[64 * v];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const uint32_t t = wave_sum(x[v].x + x[v].y + x[v].z + x[v].w);
    if (lane == 0) psum[16 * w + v] = t;
  }
#pragma unroll
  for (int v = 0; v < 16; ++v) hb[64 * v] = make_uint4(0u, 0u, 0u, 0u);
  const uint64_t r = st->rank;
  __syncthreads();   // piece totals are in LDS; every thread has read the rank
  if (w == 0) {
    const uint32_t a0 = psum[4 * lane], a1 = psum[4 * lane + 1], a2 = psum[4 * lane + 2], a3 = psum[4 * lane + 3];
    const uint32_t ls = a0 + a1 + a2 + a3;
    const uint32_t inc = wave_inclusive_scan(ls), ex = inc - ls;
    if (ex < r && r <= (uint64_t)inc) {
      uint32_t acc = ex;
      int P = 4 * lane;
      if (acc + a0 < r) {
        acc += a0; ++P;
        if (acc + a1 < r) {
          acc += a1; ++P;
          if (acc + a2 < r) { acc += a2; ++P; }
        }
      }
      pick[0] = (uint32_t)P;
      pick[1] = acc;
    }
  }
  __syncthreads();
  const uint32_t P = pick[0];
  if (P < 256 && w == (int)(P / 16)) {
    const int vs = P % 16;
    uint4 y = x[0];
#pragma unroll
    for (int v = 1; v < 16; ++v)
      if (v == vs) y = x[v];
    const uint32_t ls = y.x + y.y + y.z + y.w;
    const uint32_t inc = wave_inclusive_scan(ls);
    const uint64_t base = (uint64_t)pick[1] + (inc - ls);
    if (base < r && r <= base + ls) {
      const uint32_t c[4] = {y.x, y.y, y.z, y.w};
      uint64_t acc = base;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (acc + c[k] >= r) {
          st->rank = r - acc;
          st->prefix |= (uint64_t)(256 * P + 4 * lane + k) << shift;
          break;
        }
        acc += c[k];
      }
    }
  }
}

__global__ __launch_bounds__(1024) void k_sel_init(SelState* st, uint64_t s, uint32_t* hist) {
  if (blockIdx.x == 0 && threadIdx.x == 0) { st->prefix = 0; st->rank = s; }
  uint4* hb = reinterpret_cast<uint4*>(hist);
  for (int v = blockIdx.x * 1024 + threadIdx.x; v < SEL_BINS / 4; v += gridDim.x * 1024)
    hb[v] = make_uint4(0u, 0u, 0u, 0u);
}

__global__ __launch_bounds__(1024) void k_sel_count(int64_t M, uint64_t seed, const SelState* st,
                                                    uint32_t* __restrict__ cnt) {
  __shared__ uint32_t sh[32];
  int64_t i = (int64_t)blockIdx.x * SAMPLE_CHUNK + threadIdx.x;
  uint32_t f = (i < M && splitmix64(seed, (uint64_t)i) <= st->prefix) ? 1u : 0u;
  uint32_t tot;
  block_exclusive_scan_1024(f, sh, &tot);
  if (threadIdx.x == 0) cnt[blockIdx.x] = tot;
}

__global__ __launch_bounds__(1024) void k_sel_write(int64_t M, uint64_t seed, const SelState* st,
                                                    const uint32_t* __restrict__ off,
                                                    int32_t* __restrict__ out) {
  __shared__ uint32_t sh[32];
  int64_t i = (int64_t)blockIdx.x * SAMPLE_CHUNK + threadIdx.x;
  uint32_t f = (i < M && splitmix64(seed, (uint64_t)i) <= st->prefix) ? 1u : 0u;
  uint32_t tot;
  uint32_t ex = block_exclusive_scan_1024(f, sh, &tot);
  if (f) out[off[blockIdx.x] + ex] = (int32_t)i;
}

__global__ void k_iota(int32_t* out, int64_t n) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = (int32_t)i;
}

size_t sample_ws(int64_t M) {
  size_t nb = ceil_div(M, SAMPLE_CHUNK);
  Carve c(nullptr);
  c.take<SelState>(1);
  c.take<uint32_t>(SEL_BINS);
  c.take<uint32_t>(nb + 2);
  return c.used();
}

}  // namespace

extern "C" dsmp_status dsmp_sample_workspace(int64_t M, size_t* bytes) {
  if (!bytes || M < 0) return DSMP_INVALID_ARG;
  *bytes = sample_ws(M);
  return DSMP_OK;
}

namespace {
// The selection on a workspace of at least sample_ws(M) bytes (checked by the callers).
dsmp_status sample_run(dsmp_handle* h, int64_t M, int64_t s, uint64_t seed, int32_t* idx_out, void* ws) {
  ProfScope prof(h, DSMP_K_SAMPLE);
  if (s == M) {
    hipLaunchKernelGGL(k_iota, dim3(ceil_div(M, 256)), dim3(256), 0, h->stream, idx_out, M);
    DSMP_LAUNCHED(h, "iota");
    return DSMP_OK;
  }
  Carve c(ws);
  SelState* st = c.take<SelState>(1);
  uint32_t* hist = c.take<uint32_t>(SEL_BINS);
  int nb = (int)ceil_div(M, SAMPLE_CHUNK);
  uint32_t* cnt = c.take<uint32_t>(nb + 2);
  // the state and the histogram are cleared by a kernel on every call
  hipLaunchKernelGGL(k_sel_init, dim3(SEL_BINS / 4 / 1024), dim3(1024), 0, h->stream, st, (uint64_t)s, hist);
  unsigned g = ceil_div(M, 256);
  if (g > 2048) g = 2048;
  for (int shift = 48; shift >= 0; shift -= 16) {
    hipLaunchKernelGGL(k_sel_hist, dim3(g), dim3(256), 0, h->stream, M, seed, st, shift, hist);
    hipLaunchKernelGGL(k_sel_pick, dim3(1), dim3(1024), 0, h->stream, st, shift, hist);
  }
  hipLaunchKernelGGL(k_sel_count, dim3(nb), dim3(1024), 0, h->stream, M, seed, st, cnt);
  hipLaunchKernelGGL(k_scan_sums, dim3(1), dim3(1024), 0, h->stream, cnt, nb);
  hipLaunchKernelGGL(k_sel_write, dim3(nb), dim3(1024), 0, h->stream, M, seed, st, cnt, idx_out);
  DSMP_LAUNCHED(h, "sample");
  return DSMP_OK;
}

dsmp_status sample_check(dsmp_handle* h, int64_t M, int64_t s, const int32_t* idx_out) {
  DSMP_CHECK(h, M >= 0 && s >= 0 && s <= M, DSMP_INVALID_ARG, "need 0 <= s <= M (M=%lld s=%lld)",
             (long long)M, (long long)s);
  DSMP_CHECK(h, M <= INT32_MAX, DSMP_UNSUPPORTED, "M exceeds int32 range");
  DSMP_CHECK(h, s == 0 || idx_out != nullptr, DSMP_INVALID_ARG, "idx_out is NULL");
  return DSMP_OK;
}

// Allocation-free sampling: the workspace is a file-scope device array of a
// fixed size, enough for SAMPLE_NOALLOC_MAX_M candidates.  Host code never
// passes the array's name to a kernel: the device address comes from
// hipGetSymbolAddress, taken once per device at handle creation.
constexpr int64_t SAMPLE_NOALLOC_MAX_M = 1ll << 24;
constexpr size_t round256(size_t b) { return (b + 255) & ~size_t(255); }
constexpr size_t SAMPLE_SCRATCH_BYTES = round256(sizeof(SelState)) + round256(sizeof(uint32_t) * SEL_BINS) +
                                        round256(sizeof(uint32_t) * ((SAMPLE_NOALLOC_MAX_M + SAMPLE_CHUNK - 1) /
                                                                     SAMPLE_CHUNK + 2));
}  // namespace

static __device__ __align__(256) unsigned char scratch[SAMPLE_SCRATCH_BYTES];

static dsmp_status sample_scratch_setup(dsmp_handle* h) {
  static std::mutex mu;
  static std::map<int, void*> addr;   // device -> address of its copy of the array
  std::lock_guard<std::mutex> lock(mu);
  auto it = addr.find(h->device);
  if (it == addr.end()) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || ptr == nullptr)
      return fail(h, DSMP_HIP_ERROR, "hipGetSymbolAddress of the sampling scratch failed: %s", hipGetErrorString(e));
    it = addr.emplace(h->device, ptr).first;
  }
  h->sample_scratch = it->second;
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_sample_nodes(dsmp_handle* h, int64_t M, int64_t s, uint64_t seed,
                                         int32_t* idx_out, void* ws, size_t ws_bytes) {
  if (!h) return DSMP_INVALID_ARG;
  dsmp_status st = sample_check(h, M, s, idx_out);
  if (st != DSMP_OK || s == 0) return st;
  DSMP_CHECK(h, s == M || (ws != nullptr && ws_bytes >= sample_ws(M)), DSMP_WORKSPACE_TOO_SMALL,
             "sampling workspace needs %zu bytes", sample_ws(M));
  return sample_run(h, M, s, seed, idx_out, ws);
}

extern "C" dsmp_status dsmp_sample_nodes_noalloc(dsmp_handle* h, int64_t M, int64_t s, uint64_t seed,
                                                 int32_t* idx_out) {
  if (!h) return DSMP_INVALID_ARG;
  dsmp_status st = sample_check(h, M, s, idx_out);
  if (st != DSMP_OK || s == 0) return st;
  DSMP_CHECK(h, M <= SAMPLE_NOALLOC_MAX_M, DSMP_UNSUPPORTED,
             "allocation-free sampling takes at most %lld candidates (M=%lld)", (long long)SAMPLE_NOALLOC_MAX_M,
             (long long)M);
  DSMP_CHECK(h, h->sample_scratch != nullptr, DSMP_HIP_ERROR, "sampling scratch address not set up");
  DSMP_CHECK(h, sample_ws(M) <= SAMPLE_SCRATCH_BYTES, DSMP_UNSUPPORTED, "sampling scratch too small");
  return sample_run(h, M, s, seed, idx_out, h->sample_scratch);
}

// ------------------------------------------------------------------ gather

namespace {
__global__ void k_gather_rows(const uint32_t* __restrict__ src, int64_t n_src_rows, int64_t words,
                              const int32_t* __restrict__ idx, int64_t n, uint32_t* __restrict__ dst) {
  int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t total = n * words;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; t < total; t += stride) {
    int64_t r = t / words, w = t - r * words;
    int32_t s = idx[r];
    dst[t] = (s >= 0 && s < n_src_rows) ? src[(int64_t)s * words + w] : 0u;
  }
}
}  // namespace

extern "C" dsmp_status dsmp_gather_rows(dsmp_handle* h, const void* src, int64_t n_src_rows,
                                        int64_t row_bytes, const int32_t* idx, int64_t n, void* dst) {
  if (!h) return DSMP_INVALID_ARG;
  DSMP_CHECK(h, n >= 0 && n_src_rows >= 0 && row_bytes > 0 && row_bytes % 4 == 0, DSMP_INVALID_ARG,
             "bad gather sizes");
  if (n == 0) return DSMP_OK;
  DSMP_CHECK(h, src && idx && dst, DSMP_INVALID_ARG, "gather pointer is NULL");
  ProfScope prof(h, DSMP_K_GATHER);
  int64_t words = row_bytes / 4;
  unsigned g = ceil_div(n * words, 256);
  if (g > 8192) g = 8192;
  hipLaunchKernelGGL(k_gather_rows, dim3(g), dim3(256), 0, h->stream,
                     static_cast<const uint32_t*>(src), n_src_rows, words, idx, n,
                     static_cast<uint32_t*>(dst));
  DSMP_LAUNCHED(h, "gather_rows");
  return DSMP_OK;
}

// ------------------------------------------------------------ sub-domains

namespace {
struct Box {
  float lo[3], hi[3], elo[3], ehi[3];
};

// own[i] = 1 for nodes inside [lo, hi) in every axis; ovl[i] = 1 for the
// other nodes inside [lo - l, hi + l) (bounds rounded to float32 on the host)
__global__ void k_sub_flags(const float* __restrict__ pos, int64_t n, int D, Box b,
                            uint32_t* __restrict__ own, uint32_t* __restrict__ ovl) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  bool in = true, ext = true;
  for (int a = 0; a < D; ++a) {
    float p = pos[i * D + a];
    in = in && p >= b.lo[a] && p < b.hi[a];
    ext = ext && p >= b.elo[a] && p < b.ehi[a];
  }
  own[i] = in ? 1u : 0u;
  ovl[i] = (ext && !in) ? 1u : 0u;
}

// owned nodes to idx[0, n_owned), overlap nodes to idx[n_owned, n_total),
// each in ascending order (positions from the two exclusive scans)
__global__ void k_sub_scatter(int64_t n, const uint32_t* __restrict__ own, const uint32_t* __restrict__ ovl,
                              const int32_t* __restrict__ own_pos, const int32_t* __restrict__ ovl_pos,
                              int32_t* __restrict__ idx) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  if (own[i]) idx[own_pos[i]] = (int32_t)i;
  else if (ovl[i]) idx[own_pos[n] + ovl_pos[i]] = (int32_t)i;
}

__global__ void k_scatter_rows(const uint32_t* __restrict__ src, int64_t words, const int32_t* __restrict__ idx,
                               int64_t n, uint32_t* __restrict__ dst, int64_t n_dst_rows) {
  int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t total = n * words;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; t < total; t += stride) {
    int64_t r = t / words, w = t - r * words;
    int32_t d = idx[r];
    if (d >= 0 && d < n_dst_rows) dst[(int64_t)d * words + w] = src[t];
  }
}

struct SubWs {
  uint32_t *own, *ovl, *tmp;
  int32_t *own_pos, *ovl_pos;
};

SubWs carve_sub(void* ws, int64_t n, size_t* used) {
  Carve c(ws);
  SubWs w;
  w.own = c.take<uint32_t>(n + 1);
  w.ovl = c.take<uint32_t>(n + 1);
  w.own_pos = c.take<int32_t>(n + 1);
  w.ovl_pos = c.take<int32_t>(n + 1);
  w.tmp = c.take<uint32_t>(scan_tmp_elems(n));
  *used = c.used();
  return w;
}
}  // namespace

extern "C" dsmp_status dsmp_subdomain_workspace(int64_t n, size_t* bytes) {
  if (!bytes || n < 0) return DSMP_INVALID_ARG;
  carve_sub(nullptr, n, bytes);
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_subdomain_select(dsmp_handle* h, const float* pos, int64_t n, int32_t dim,
                                             const float* lo, const float* hi, float overlap,
                                             int32_t* idx_out, void* ws, size_t ws_bytes,
                                             int64_t* n_owned, int64_t* n_total) {
  if (!h) return DSMP_INVALID_ARG;
  DSMP_CHECK(h, n >= 0 && n <= INT32_MAX, n < 0 ? DSMP_INVALID_ARG : DSMP_UNSUPPORTED, "bad node count");
  DSMP_CHECK(h, dim == 2 || dim == 3, DSMP_UNSUPPORTED, "dim must be 2 or 3");
  DSMP_CHECK(h, lo && hi && n_owned && n_total, DSMP_INVALID_ARG, "sub-domain pointer is NULL");
  DSMP_CHECK(h, overlap >= 0.0f, DSMP_INVALID_ARG, "overlap must be >= 0");
  *n_owned = 0;
  *n_total = 0;
  if (n == 0) return DSMP_OK;
  DSMP_CHECK(h, pos && idx_out && ws, DSMP_INVALID_ARG, "sub-domain pointer is NULL");
  size_t need;
  SubWs w = carve_sub(ws, n, &need);
  DSMP_CHECK(h, ws_bytes >= need, DSMP_WORKSPACE_TOO_SMALL, "sub-domain workspace %zu < %zu", ws_bytes, need);
  Box b{};
  for (int a = 0; a < dim; ++a) {
    b.lo[a] = lo[a];
    b.hi[a] = hi[a];
    b.elo[a] = lo[a] - overlap;   // float32 rounding, as the bounds are defined
    b.ehi[a] = hi[a] + overlap;
  }
  ProfScope prof(h, DSMP_K_GATHER);
  hipStream_t s = h->stream;
  hipLaunchKernelGGL(k_sub_flags, dim3(ceil_div(n, 256)), dim3(256), 0, s, pos, n, (int)dim, b, w.own, w.ovl);
  DSMP_LAUNCHED(h, "sub-domain flags");
  dsmp_status st;
  if ((st = exclusive_scan_u32(h, w.own, w.own_pos, n, w.tmp)) != DSMP_OK) return st;
  if ((st = exclusive_scan_u32(h, w.ovl, w.ovl_pos, n, w.tmp)) != DSMP_OK) return st;
  hipLaunchKernelGGL(k_sub_scatter, dim3(ceil_div(n, 256)), dim3(256), 0, s, n, w.own, w.ovl, w.own_pos,
                     w.ovl_pos, idx_out);
  DSMP_LAUNCHED(h, "sub-domain scatter");
  int32_t tot[2];
  DSMP_HIP(h, hipMemcpyAsync(&tot[0], w.own_pos + n, sizeof(int32_t), hipMemcpyDeviceToHost, s));
  DSMP_HIP(h, hipMemcpyAsync(&tot[1], w.ovl_pos + n, sizeof(int32_t), hipMemcpyDeviceToHost, s));
  DSMP_HIP(h, hipStreamSynchronize(s));
  *n_owned = tot[0];
  *n_total = (int64_t)tot[0] + tot[1];
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_scatter_rows(dsmp_handle* h, const void* src, int64_t n, int64_t row_bytes,
                                         const int32_t* idx, void* dst, int64_t n_dst_rows) {
  if (!h) return DSMP_INVALID_ARG;
  DSMP_CHECK(h, n >= 0 && n_dst_rows >= 0 && row_bytes > 0 && row_bytes % 4 == 0, DSMP_INVALID_ARG,
             "bad scatter sizes");
  if (n == 0) return DSMP_OK;
  DSMP_CHECK(h, src && idx && dst, DSMP_INVALID_ARG, "scatter pointer is NULL");
  ProfScope prof(h, DSMP_K_GATHER);
  int64_t words = row_bytes / 4;
  unsigned g = ceil_div(n * words, 256);
  if (g > 8192) g = 8192;
  hipLaunchKernelGGL(k_scatter_rows, dim3(g), dim3(256), 0, h->stream, static_cast<const uint32_t*>(src), words,
                     idx, n, static_cast<uint32_t*>(dst), n_dst_rows);
  DSMP_LAUNCHED(h, "scatter_rows");
  return DSMP_OK;
}
