// Radius-graph kernels (Sec. 2.1; Algorithm 1, edge-index creation and edge
// sampling): uniform-grid cell hash, counting sort of the points into cells,
// per-destination neighbour count, scan to CSR, neighbour fill with the edge
// cap, and the source-grouped transpose.
//
// Determinism: integer atomics are used only for counts and slot claims; every
// row is sorted before it is written, so the order in which candidates were
// visited never reaches the output.
//
// Built with -ffp-contract=off; the distance test also spells out its
// roundings with __fsub_rn / __fmul_rn / __fadd_rn.
#include "common.hpp"

using namespace dsmp;

namespace {

constexpr int ROW_LIMIT = 4096;   // most sources within r of one destination
constexpr int BBOX_BLOCKS = 256;

struct GridParams {
  float lo[3];
  int dims[3];
  int ncell;
  double inv_c;   // 1 / cell width
};

struct GraphStats {
  unsigned long long total;   // sum of kept counts (64-bit, for the overflow check)
  unsigned int maxraw;        // largest pre-cap count of a row
  unsigned int pad;
};

__device__ __forceinline__ float3 load_pos(const float* __restrict__ pos, int64_t i, int D) {
  const float* p = pos + i * D;
  return make_float3(p[0], p[1], D == 3 ? p[2] : 0.0f);
}

// canonical float32 squared distance: no contraction, fixed order
__device__ __forceinline__ float dist2(float3 a, float3 b, int D) {
  float dx = __fsub_rn(b.x, a.x);
  float dy = __fsub_rn(b.y, a.y);
  float d2 = __fadd_rn(__fmul_rn(dx, dx), __fmul_rn(dy, dy));
  if (D == 3) {
    float dz = __fsub_rn(b.z, a.z);
    d2 = __fadd_rn(d2, __fmul_rn(dz, dz));
  }
  return d2;
}

__global__ __launch_bounds__(256) void k_bbox_partial(const float* __restrict__ pos, int64_t n, int D,
                                                      float* __restrict__ part) {
  __shared__ float sh[6][256];
  float mn[3] = {INFINITY, INFINITY, INFINITY}, mx[3] = {-INFINITY, -INFINITY, -INFINITY};
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    float3 p = load_pos(pos, i, D);
    float v[3] = {p.x, p.y, p.z};
    for (int a = 0; a < 3; ++a) { mn[a] = fminf(mn[a], v[a]); mx[a] = fmaxf(mx[a], v[a]); }
  }
  for (int a = 0; a < 3; ++a) { sh[a][threadIdx.x] = mn[a]; sh[3 + a][threadIdx.x] = mx[a]; }
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s)
      for (int a = 0; a < 3; ++a) {
        sh[a][threadIdx.x] = fminf(sh[a][threadIdx.x], sh[a][threadIdx.x + s]);
        sh[3 + a][threadIdx.x] = fmaxf(sh[3 + a][threadIdx.x], sh[3 + a][threadIdx.x + s]);
      }
    __syncthreads();
  }
  if (threadIdx.x < 6) part[blockIdx.x * 6 + threadIdx.x] = sh[threadIdx.x][0];
}

// One wave reduces the partial boxes, one lane chooses the cell size.  Cells are
// at least r*(1 + 2^-10) wide, so two points that pass the float32 radius
// test always sit in the same or adjacent cells (cell coordinates are formed
// in double, see cell_coord); the grid is coarsened by doubling until it has
// at most `cap` cells.
__global__ void k_grid_setup(const float* __restrict__ part, int nb, int D, float r, int64_t cap,
                             GridParams* __restrict__ g, GraphStats* __restrict__ st) {
  const int lane = threadIdx.x;  // one wave
  float lo[3] = {INFINITY, INFINITY, INFINITY}, hi[3] = {-INFINITY, -INFINITY, -INFINITY};
  for (int b = lane; b < nb; b += 64)
    for (int a = 0; a < 3; ++a) {
      lo[a] = fminf(lo[a], part[b * 6 + a]);
      hi[a] = fmaxf(hi[a], part[b * 6 + 3 + a]);
    }
  for (int o = 32; o > 0; o >>= 1)
    for (int a = 0; a < 3; ++a) {
      lo[a] = fminf(lo[a], __shfl_xor(lo[a], o, 64));
      hi[a] = fmaxf(hi[a], __shfl_xor(hi[a], o, 64));
    }
  if (lane != 0) return;
  for (int a = D; a < 3; ++a) { lo[a] = 0.0f; hi[a] = 0.0f; }
  for (int a = 0; a < 3; ++a)
    if (!(hi[a] >= lo[a])) { lo[a] = 0.0f; hi[a] = 0.0f; }   // empty input
  double c = (double)r * (1.0 + 1.0 / 1024.0);
  if (!(c > 1e-30)) c = 1e-30;
  double dims[3];
  for (;;) {
    double cells = 1.0;
    for (int a = 0; a < 3; ++a) {
      dims[a] = floor(((double)hi[a] - (double)lo[a]) / c) + 1.0;
      cells *= dims[a];
    }
    if (cells <= (double)cap) break;
    c *= 2.0;
  }
  for (int a = 0; a < 3; ++a) { g->lo[a] = lo[a]; g->dims[a] = (int)dims[a]; }
  g->inv_c = 1.0 / c;
  g->ncell = g->dims[0] * g->dims[1] * g->dims[2];
  st->total = 0;
  st->maxraw = 0;
}

// Cell of coordinate v, in double: v - lo is exact there and the product
// with 1/c is within 2^-52 of the cell coordinate, so the cell margin of
// 2^-10 covers the rounding however many cells an axis has (in float32 the
// worst-case error grows with the coordinate and reaches the margin at a few
// thousand cells on an axis, which a long, thin point set can have).
__device__ __forceinline__ int cell_coord(float v, float lo, double inv_c, int dim) {
  const double t = ((double)v - (double)lo) * inv_c;
  int c = (int)floor(t);
  return c < 0 ? 0 : (c >= dim ? dim - 1 : c);
}

__global__ __launch_bounds__(256) void k_cell_hash(const float* __restrict__ pos, int64_t n, int D,
                                                   const GridParams* __restrict__ g,
                                                   uint32_t* __restrict__ cellid,
                                                   uint32_t* __restrict__ ccount) {
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  float3 p = load_pos(pos, i, D);
  int cx = cell_coord(p.x, g->lo[0], g->inv_c, g->dims[0]);
  int cy = cell_coord(p.y, g->lo[1], g->inv_c, g->dims[1]);
  int cz = D == 3 ? cell_coord(p.z, g->lo[2], g->inv_c, g->dims[2]) : 0;
  uint32_t id = (uint32_t)(cx + g->dims[0] * (cy + g->dims[1] * cz));
  cellid[i] = id;
  atomicAdd(&ccount[id], 1u);
}

__global__ __launch_bounds__(256) void k_cell_scatter(const float* __restrict__ pos, int64_t n, int D,
                                                      const uint32_t* __restrict__ cellid,
                                                      const int32_t* __restrict__ cstart,
                                                      uint32_t* __restrict__ cur,
                                                      float4* __restrict__ spos,
                                                      int32_t* __restrict__ sidx) {
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  uint32_t c = cellid[i];
  int32_t slot = cstart[c] + (int32_t)atomicAdd(&cur[c], 1u);
  float3 p = load_pos(pos, i, D);
  spos[slot] = make_float4(p.x, p.y, p.z, 0.0f);
  sidx[slot] = (int32_t)i;
}

// The candidates of a destination: for every neighbouring cell row (3 in 2-D,
// 9 in 3-D) the three cells along x are one contiguous range of the
// cell-sorted arrays. Lane k < 9 loads the bounds of range k, so that all of
// them are in flight at once; the ranges are then numbered as one flat list of
// `total` candidates (wave-uniform starts a[k] and flat offsets off[k]).
struct Candidates {
  int a[9];
  int off[9];
  int total;
};

__device__ __forceinline__ Candidates candidate_ranges(float3 p, int D, const GridParams& g,
                                                       const int32_t* __restrict__ cstart,
                                                       int lane) {
  const int cx = cell_coord(p.x, g.lo[0], g.inv_c, g.dims[0]);
  const int cy = cell_coord(p.y, g.lo[1], g.inv_c, g.dims[1]);
  const int cz = D == 3 ? cell_coord(p.z, g.lo[2], g.inv_c, g.dims[2]) : 0;
  const int x0 = cx > 0 ? cx - 1 : 0, x1 = cx + 1 < g.dims[0] ? cx + 1 : g.dims[0] - 1;
  const int nr = D == 3 ? 9 : 3;
  int a = 0, len = 0;
  if (lane < nr) {
    const int z = cz + (D == 3 ? lane / 3 - 1 : 0);
    const int y = cy + lane % 3 - 1;
    if (z >= 0 && z < g.dims[2] && y >= 0 && y < g.dims[1]) {
      const int base = g.dims[0] * (y + g.dims[1] * z);
      a = cstart[base + x0];
      len = cstart[base + x1 + 1] - a;
    }
  }
  int inc = len;  // inclusive prefix over lanes 0..15 (lanes past nr hold 0)
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) {
    const int v = __shfl_up(inc, o, 64);
    if (lane >= o) inc += v;
  }
  Candidates c;
#pragma unroll
  for (int k = 0; k < 9; ++k) {
    c.a[k] = __builtin_amdgcn_readlane(a, k);
    c.off[k] = __builtin_amdgcn_readlane(inc - len, k);
  }
  c.total = __builtin_amdgcn_readlane(inc, 15);
  return c;
}

// Position in the cell-sorted arrays of flat candidate t (0 <= t < total).
// Offsets never decrease, so the last range whose offset is at most t holds it.
__device__ __forceinline__ int candidate_at(const Candidates& c, int t) {
  int s = c.a[0] + t;
#pragma unroll
  for (int k = 1; k < 9; ++k)
    if (t >= c.off[k]) s = c.a[k] + (t - c.off[k]);
  return s;
}

// Candidates are read CAND_BATCHES x 64 at a time, all loads issued before the
// first test.
constexpr int CAND_BATCHES = 4;

// Calls f(t, q, j) for every flat candidate t of a destination, with its
// position and source index; lanes past the end get t >= total. Every lane of
// the wave calls f the same number of times.
template <typename F>
__device__ __forceinline__ void for_each_candidate(const Candidates& c, int lane,
                                                   const float4* __restrict__ spos,
                                                   const int32_t* __restrict__ sidx, F f) {
  for (int t0 = 0; t0 < c.total; t0 += 64 * CAND_BATCHES) {
    float4 q[CAND_BATCHES];
    int32_t j[CAND_BATCHES];
#pragma unroll
    for (int u = 0; u < CAND_BATCHES; ++u) {
      const int t = t0 + 64 * u + lane;
      const int sidx_pos = candidate_at(c, t < c.total ? t : c.total - 1);
      q[u] = spos[sidx_pos];
      j[u] = sidx[sidx_pos];
    }
#pragma unroll
    for (int u = 0; u < CAND_BATCHES; ++u) f(t0 + 64 * u + lane, q[u], j[u]);
  }
}

// One wave per destination row: count the sources that pass the radius test.
__global__ __launch_bounds__(256) void k_nbr_count(const float* __restrict__ pos, int64_t n_dst, int D,
                                                   float r2, int cap, const GridParams* __restrict__ gp,
                                                   const int32_t* __restrict__ cstart,
                                                   const float4* __restrict__ spos,
                                                   const int32_t* __restrict__ sidx,
                                                   uint32_t* __restrict__ rcnt,
                                                   uint32_t* __restrict__ rraw) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= n_dst) return;
  const GridParams g = *gp;
  const float3 pi = load_pos(pos, i, D);
  const Candidates c = candidate_ranges(pi, D, g, cstart, lane);
  uint32_t cnt = 0;
  for_each_candidate(c, lane, spos, sidx, [&](int t, float4 q, int32_t j) {
    const float d2 = dist2(pi, make_float3(q.x, q.y, q.z), D);
    if (t < c.total && d2 <= r2 && j != (int32_t)i) ++cnt;
  });
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
  if (lane == 0) {
    rcnt[i] = (cap > 0 && cnt > (uint32_t)cap) ? (uint32_t)cap : cnt;
    rraw[i] = cnt;
  }
}

// Edge total (64-bit) and largest pre-cap row count: every block reduces a
// strided share of the rows and adds its result atomically (grid setup has
// zeroed both).
__global__ __launch_bounds__(256) void k_graph_stats(const uint32_t* __restrict__ rcnt,
                                                     const uint32_t* __restrict__ rraw, int64_t n_dst,
                                                     GraphStats* __restrict__ st) {
  __shared__ unsigned long long ssum[4];
  __shared__ uint32_t smax[4];
  unsigned long long s = 0;
  uint32_t m = 0;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n_dst; i += (int64_t)gridDim.x * 256) {
    s += rcnt[i];
    m = rraw[i] > m ? rraw[i] : m;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    s += __shfl_xor(s, o, 64);
    const uint32_t v = __shfl_xor(m, o, 64);
    m = v > m ? v : m;
  }
  if ((threadIdx.x & 63) == 0) {
    ssum[threadIdx.x >> 6] = s;
    smax[threadIdx.x >> 6] = m;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    s = ssum[0] + ssum[1] + ssum[2] + ssum[3];
    m = smax[0];
    for (int k = 1; k < 4; ++k) m = smax[k] > m ? smax[k] : m;
    atomicAdd(&st->total, s);
    atomicMax(&st->maxraw, m);
  }
}

// Orders shared-memory accesses between the lanes of one wave: the rows a
// block holds are independent waves, each with its own slice of shared
// memory, so they never wait for each other.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Bitonic sort of P (power of two) 64-bit keys with 32-bit payload, by one wave.
__device__ void bitonic_kv(uint64_t* key, int32_t* val, int P, int lane) {
  for (int k = 2; k <= P; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int t = lane; t < P; t += 64) {
        int u = t ^ j;
        if (u > t) {
          bool up = (t & k) == 0;
          uint64_t a = key[t], b = key[u];
          if ((a > b) == up) {
            key[t] = b; key[u] = a;
            int32_t v = val[t]; val[t] = val[u]; val[u] = v;
          }
        }
      }
      wave_sync();
    }
}

__device__ void bitonic_u32(uint32_t* key, int P, int lane) {
  for (int k = 2; k <= P; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int t = lane; t < P; t += 64) {
        int u = t ^ j;
        if (u > t) {
          bool up = (t & k) == 0;
          uint32_t a = key[t], b = key[u];
          if ((a > b) == up) { key[t] = b; key[u] = a; }
        }
      }
      wave_sync();
    }
}

// Place of each lane's value among the first n lanes' values (n <= 64,
// values distinct): the number of smaller ones.
__device__ __forceinline__ int wave_rank(uint32_t v, int n) {
  int rank = 0;
  for (int k = 0; k < n; ++k) rank += (uint32_t)__builtin_amdgcn_readlane((int)v, k) < v;
  return rank;
}

__device__ __forceinline__ int next_pow2(int n) {
  int p = 1;
  while (p < n) p <<= 1;
  return p;
}

// Rows of up to 64 SEL_PER_LANE candidates take the cap by a radix select in
// registers; longer rows sort their keys in LDS.
constexpr int SEL_PER_LANE = 8;

// The one-pass select of capped graphs: caps up to FUSE_CAP, rows of up to
// FUSE_LIM candidates (larger rows are built by the fill kernel).
constexpr int FUSE_CAP = 64;
constexpr int FUSE_LIM = 256;

// Writes to js the payloads of the cap smallest of the n keys (cap < n <=
// 64 NT) without sorting them. Keys are distinct: d2 bits with the source
// index, or a bijective hash of a distinct counter. The cap-th smallest key K
// is fixed bit by bit from the top (a radix select over the keys held in
// registers, NT per lane, with counts by ballots) until one key alone matches
// the fixed bits; the kept keys are those whose fixed bits are at most K's.
// The high words decide unless two of them are equal at K; only then are the
// low words visited.
template <int NT>
__device__ __forceinline__ void select_cap(const uint64_t* key, const int32_t* val, uint32_t* js,
                                           int n, int cap, int lane) {
  uint32_t kh[NT], kl[NT];
  int32_t vr[NT];
  uint64_t vm[NT];  // lanes that hold a key (wave-uniform)
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int u = lane + 64 * t;
    const bool ok = u < n;
    const uint64_t k = ok ? key[u] : ~0ull;
    kh[t] = (uint32_t)(k >> 32);
    kl[t] = (uint32_t)k;
    vr[t] = ok ? val[u] : 0;
    vm[t] = __ballot(ok);
  }
  int rank = cap - 1;  // K's rank among the keys that match the fixed bits
  int tot = n;         // how many keys match them
  uint32_t mh = 0, ph = 0, ml = 0, pl = 0;  // fixed bits of K (masks) and their values
  for (int b = 31; b >= 0 && tot > 1; --b) {
    const uint32_t sel = mh | (1u << b);  // bit b of ph is still clear
    int c = 0;  // matching keys with bit b clear
#pragma unroll
    for (int t = 0; t < NT; ++t) c += __popcll(__ballot(((kh[t] ^ ph) & sel) == 0) & vm[t]);
    if (rank >= c) {
      ph |= 1u << b;
      rank -= c;
      tot -= c;
    } else {
      tot = c;
    }
    mh = sel;
  }
  for (int b = 31; b >= 0 && tot > 1; --b) {
    const uint32_t sel = ml | (1u << b);
    int c = 0;
#pragma unroll
    for (int t = 0; t < NT; ++t)
      c += __popcll(__ballot(kh[t] == ph && ((kl[t] ^ pl) & sel) == 0) & vm[t]);
    if (rank >= c) {
      pl |= 1u << b;
      rank -= c;
      tot -= c;
    } else {
      tot = c;
    }
    ml = sel;
  }
  wave_sync();  // every key is read; js overwrites them
  int m0 = 0;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const uint32_t h = kh[t] & mh;
    const bool keep = h < ph || (h == ph && (kl[t] & ml) <= pl);
    const uint64_t bm = __ballot(keep) & vm[t];
    const int slot = m0 + __popcll(bm & ((1ull << lane) - 1ull));
    if (((bm >> lane) & 1ull) && slot < cap) js[slot] = (uint32_t)vr[t];
    m0 += __popcll(bm);
  }
}

// One wave per destination row, up to four rows per block (each wave with
// its own lim x 12 bytes of shared memory): gather the sources that pass the
// test, apply the cap (the cap smallest keys: (d2, j) or the hashed key), sort
// the kept sources by index and write the row. When indeg is given, every
// written edge also adds one to its source's in-degree. When rraw is given,
// only rows with more than raw_above candidates are filled.
__global__ __launch_bounds__(256) void k_nbr_fill(const float* __restrict__ pos, int64_t n_dst,
                                                  int64_t n_src, int D, float r2, int cap,
                                                  int cap_mode, uint64_t seed, int lim,
                                                  const GridParams* __restrict__ gp,
                                                  const int32_t* __restrict__ cstart,
                                                  const float4* __restrict__ spos,
                                                  const int32_t* __restrict__ sidx,
                                                  const int32_t* __restrict__ row_ptr,
                                                  int64_t capacity, int32_t* __restrict__ col,
                                                  int32_t* __restrict__ dst,
                                                  uint32_t* __restrict__ indeg,
                                                  const uint32_t* __restrict__ rraw, int raw_above) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int wv = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  uint64_t* key = reinterpret_cast<uint64_t*>(smem + (size_t)wv * lim * 12);
  int32_t* val = reinterpret_cast<int32_t*>(smem + (size_t)wv * lim * 12 + (size_t)lim * 8);
  const int64_t i = (int64_t)blockIdx.x * (blockDim.x >> 6) + wv;
  if (i >= n_dst) return;
  if (rraw && rraw[i] <= (uint32_t)raw_above) return;  // placed from the select's slab
  const int64_t base = row_ptr[i];
  const GridParams g = *gp;
  const float3 pi = load_pos(pos, i, D);
  const Candidates c = candidate_ranges(pi, D, g, cstart, lane);
  int n = 0;
  for_each_candidate(c, lane, spos, sidx, [&](int t, float4 q, int32_t j) {
    const float d2 = dist2(pi, make_float3(q.x, q.y, q.z), D);
    const bool pass = t < c.total && d2 <= r2 && j != (int32_t)i;
    const uint64_t m = __ballot(pass);
    if (pass) {
      const int slot = n + __popcll(m & ((1ull << lane) - 1ull));
      const uint64_t k = cap_mode == DSMP_CAP_KNN
                             ? (((uint64_t)__float_as_uint(d2)) << 32) | (uint32_t)j
                             : splitmix64(seed, (uint64_t)i * (uint64_t)n_src + (uint64_t)j);
      if (slot < lim) {
        key[slot] = k;
        val[slot] = j;
      }
    }
    n += __popcll(m);
  });
  n = n < lim ? n : lim;
  wave_sync();
  uint32_t* js = reinterpret_cast<uint32_t*>(key);   // kept sources (the key array reused as uint32 scratch)
  if (cap > 0 && n > cap && n <= 64 * SEL_PER_LANE) {
    switch ((n + 63) >> 6) {
      case 1: select_cap<1>(key, val, js, n, cap, lane); break;
      case 2: select_cap<2>(key, val, js, n, cap, lane); break;
      case 3: select_cap<3>(key, val, js, n, cap, lane); break;
      case 4: select_cap<4>(key, val, js, n, cap, lane); break;
      case 5: select_cap<5>(key, val, js, n, cap, lane); break;
      case 6: select_cap<6>(key, val, js, n, cap, lane); break;
      case 7: select_cap<7>(key, val, js, n, cap, lane); break;
      default: select_cap<8>(key, val, js, n, cap, lane); break;
    }
    n = cap;
  } else {
    if (cap > 0 && n > cap) {
      int P = next_pow2(n);
      for (int t = n + lane; t < P; t += 64) { key[t] = ~0ull; val[t] = INT32_MAX; }
      wave_sync();
      bitonic_kv(key, val, P, lane);
      n = cap;
    }
    for (int t = lane; t < n; t += 64) js[t] = (uint32_t)val[t];
  }
  wave_sync();
  if (n <= 64) {
    // Rows of up to 64 kept sources are sorted in registers (the indices of
    // a row are distinct).
    const uint32_t mj = lane < n ? js[lane] : 0xFFFFFFFFu;
    const int64_t e = base + wave_rank(mj, n);
    if (lane < n && e < capacity) {
      col[e] = (int32_t)mj;
      dst[e] = (int32_t)i;
      if (indeg) atomicAdd(&indeg[mj], 1u);
    }
    return;
  }
  int P = next_pow2(n);
  for (int t = n + lane; t < P; t += 64) js[t] = 0xFFFFFFFFu;
  wave_sync();
  bitonic_u32(js, P, lane);
  for (int t = lane; t < n; t += 64) {
    int64_t e = base + t;
    if (e < capacity) {
      col[e] = (int32_t)js[t];
      dst[e] = (int32_t)i;
      if (indeg) atomicAdd(&indeg[js[t]], 1u);
    }
  }
}

__global__ __launch_bounds__(256) void k_csc_scatter(const int32_t* __restrict__ col, int64_t E,
                                                     const int32_t* __restrict__ csc_ptr,
                                                     uint32_t* __restrict__ cur,
                                                     int32_t* __restrict__ csc_eid) {
  int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= E) return;
  int32_t j = col[e];
  csc_eid[csc_ptr[j] + (int32_t)atomicAdd(&cur[j], 1u)] = (int32_t)e;
}

// Uncapped graph over one point set (n_src = n_dst, no cap): j is a source of
// i exactly when i is a source of j (the float32 distance test is symmetric,
// fl(a - b) = -fl(b - a)), so the edges leaving j are the edges (i <- j) for i
// in row j, in row order, which is ascending edge id: csc_ptr = row_ptr, and
// position e of row j holds the id of edge (col[e] <- j), row_ptr[i] + the
// position of j in row i (rows are sorted by source).
// The same launch copies row_ptr (n_ptr entries) to csc_ptr.
__global__ __launch_bounds__(256) void k_csc_symmetric(const int32_t* __restrict__ row_ptr, int64_t n_ptr,
                                                       const int32_t* __restrict__ col,
                                                       const int32_t* __restrict__ dst, int64_t E,
                                                       int32_t* __restrict__ csc_ptr,
                                                       int32_t* __restrict__ csc_eid) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < n_ptr) csc_ptr[e] = row_ptr[e];
  if (e >= E) return;
  const int32_t i = col[e], j = dst[e];
  int32_t lo = row_ptr[i], hi = row_ptr[i + 1];   // first position in row i with col >= j
  while (lo < hi) {
    const int32_t mid = lo + (hi - lo) / 2;
    if (col[mid] < j) lo = mid + 1;
    else hi = mid;
  }
  csc_eid[e] = lo;
}

constexpr int CSC_SORT_LDS = 2048;

// One wave per source: sort its edge ids ascending (LDS bitonic; an in-place
// insertion sort by one lane for the rare longer groups).
// Sorts each source's incoming edge ids. A wave takes CSC_COLS consecutive
// sources (their loads issued together), four waves per block: up to 64 ids
// are sorted in registers, up to CSC_SORT_LDS in shared memory, longer
// columns by one lane.
constexpr int CSC_COLS = 4;

__global__ __launch_bounds__(256) void k_csc_sort(const int32_t* __restrict__ csc_ptr, int64_t n_src,
                                                  int32_t* __restrict__ csc_eid) {
  __shared__ uint32_t sbuf[4][CSC_SORT_LDS];
  const int wv = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int64_t j0 = ((int64_t)blockIdx.x * 4 + wv) * CSC_COLS;
  if (j0 >= n_src) return;
  uint32_t* buf = sbuf[wv];
  int ptr[CSC_COLS + 1];
#pragma unroll
  for (int c = 0; c <= CSC_COLS; ++c) ptr[c] = csc_ptr[j0 + c < n_src ? j0 + c : n_src];
  uint32_t v[CSC_COLS];
#pragma unroll
  for (int c = 0; c < CSC_COLS; ++c) {
    // in bounds for every lane: the column's own ids, else the first edge
    const int n = ptr[c + 1] - ptr[c];
    const int at = n > 0 ? ptr[c] + (lane < n ? lane : n - 1) : 0;
    const uint32_t x = (uint32_t)csc_eid[at];
    v[c] = lane < n ? x : 0xFFFFFFFFu;
  }
#pragma unroll
  for (int c = 0; c < CSC_COLS; ++c) {
    const int a = ptr[c], b = ptr[c + 1], n = b - a;
    if (n <= 1) continue;
    if (n <= 64) {
      const int rank = wave_rank(v[c], n);
      if (lane < n) csc_eid[a + rank] = (int32_t)v[c];
    } else if (n <= CSC_SORT_LDS) {
      int P = next_pow2(n);
      for (int t = lane; t < P; t += 64) buf[t] = t < n ? (uint32_t)csc_eid[a + t] : 0xFFFFFFFFu;
      wave_sync();
      bitonic_u32(buf, P, lane);
      for (int t = lane; t < n; t += 64) csc_eid[a + t] = (int32_t)buf[t];
      wave_sync();  // buf is free for the next column
    } else if (lane == 0) {
      for (int t = a + 1; t < b; ++t) {
        int32_t x = csc_eid[t];
        int u = t - 1;
        while (u >= a && csc_eid[u] > x) { csc_eid[u + 1] = csc_eid[u]; --u; }
        csc_eid[u + 1] = x;
      }
    }
  }
}

// One pass per row for capped graphs: gather the sources that pass the test,
// keep the cap smallest keys and write them, sorted by index, to the row's cap
// slots of the slab; count the row, and each kept edge into its source's
// in-degree (zeroed beforehand), keeping the count it found there as the
// edge's place among its source's edges (in no fixed order; the transpose is
// sorted afterwards). One wave per row, four per block, each
// wave with room for FUSE_LIM candidates: a row with more is only counted
// (the fill kernel builds it after the scan).
__global__ __launch_bounds__(256) void k_nbr_select(const float* __restrict__ pos, int64_t n_dst,
                                                    int64_t n_src, int D, float r2, int cap,
                                                    int cap_mode, uint64_t seed,
                                                    const GridParams* __restrict__ gp,
                                                    const int32_t* __restrict__ cstart,
                                                    const float4* __restrict__ spos,
                                                    const int32_t* __restrict__ sidx,
                                                    uint32_t* __restrict__ rcnt,
                                                    uint32_t* __restrict__ rraw,
                                                    uint32_t* __restrict__ slab,
                                                    uint32_t* __restrict__ indeg,
                                                    uint32_t* __restrict__ eslot) {
  __shared__ uint64_t skey[4][FUSE_LIM];
  __shared__ int32_t sval[4][FUSE_LIM];
  const int wv = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * 4 + wv;
  if (i >= n_dst) return;
  uint64_t* key = skey[wv];
  int32_t* val = sval[wv];
  const GridParams g = *gp;
  const float3 pi = load_pos(pos, i, D);
  const Candidates c = candidate_ranges(pi, D, g, cstart, lane);
  int n = 0;
  for_each_candidate(c, lane, spos, sidx, [&](int t, float4 q, int32_t j) {
    const float d2 = dist2(pi, make_float3(q.x, q.y, q.z), D);
    const bool pass = t < c.total && d2 <= r2 && j != (int32_t)i;
    const uint64_t m = __ballot(pass);
    if (pass) {
      const int slot = n + __popcll(m & ((1ull << lane) - 1ull));
      if (slot < FUSE_LIM) {
        key[slot] = cap_mode == DSMP_CAP_KNN
                        ? (((uint64_t)__float_as_uint(d2)) << 32) | (uint32_t)j
                        : splitmix64(seed, (uint64_t)i * (uint64_t)n_src + (uint64_t)j);
        val[slot] = j;
      }
    }
    n += __popcll(m);
  });
  const int kept = n < cap ? n : cap;
  if (lane == 0) {
    rraw[i] = (uint32_t)n;
    rcnt[i] = (uint32_t)kept;
  }
  if (n > FUSE_LIM) return;
  wave_sync();
  uint32_t* js = reinterpret_cast<uint32_t*>(key);  // kept sources, over the keys
  if (n > cap) {
    switch ((n + 63) >> 6) {
      case 1: select_cap<1>(key, val, js, n, cap, lane); break;
      case 2: select_cap<2>(key, val, js, n, cap, lane); break;
      case 3: select_cap<3>(key, val, js, n, cap, lane); break;
      default: select_cap<4>(key, val, js, n, cap, lane); break;
    }
  } else {
    for (int t = lane; t < n; t += 64) js[t] = (uint32_t)val[t];
  }
  wave_sync();
  // kept <= cap <= 64: sorted in registers
  const uint32_t mj = lane < kept ? js[lane] : 0xFFFFFFFFu;
  const int rank = wave_rank(mj, kept);
  if (lane < kept) {
    slab[i * cap + rank] = mj;
    eslot[i * cap + rank] = atomicAdd(&indeg[mj], 1u);
  }
}

// Copies the selected rows from the slab into the CSR arrays, one thread per
// slab entry, and, given csc_ptr, each edge id into its source's column at the
// place the select found. Rows with more than FUSE_LIM candidates are left to
// the fill kernel.
__global__ __launch_bounds__(256) void k_nbr_place(int64_t n_dst, int cap, const uint32_t* __restrict__ rraw,
                                                   const int32_t* __restrict__ row_ptr,
                                                   const uint32_t* __restrict__ slab,
                                                   const uint32_t* __restrict__ eslot,
                                                   const int32_t* __restrict__ csc_ptr, int64_t capacity,
                                                   int32_t* __restrict__ col, int32_t* __restrict__ dst,
                                                   int32_t* __restrict__ csc_eid) {
  const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (x >= n_dst * cap) return;
  const int64_t i = x / cap;
  const int t = (int)(x - i * cap);
  if (rraw[i] > (uint32_t)FUSE_LIM) return;
  const int64_t base = row_ptr[i];
  const int64_t e = base + t;
  if (e < row_ptr[i + 1] && e < capacity) {
    const uint32_t j = slab[x];
    col[e] = (int32_t)j;
    dst[e] = (int32_t)i;
    if (csc_ptr) {
      const int64_t p = (int64_t)csc_ptr[j] + eslot[x];
      if (p < capacity) csc_eid[p] = (int32_t)e;
    }
  }
}

struct GraphWs {
  float* part;
  GridParams* grid;
  GraphStats* stats;
  uint32_t* cellid;
  uint32_t* ccount;
  int32_t* cstart;
  uint32_t* ccur;
  float4* spos;
  int32_t* sidx;
  uint32_t* rcnt;
  uint32_t* rraw;
  int32_t* rowptr_tmp;
  uint32_t* indeg;
  uint32_t* scur;
  uint32_t* scan_tmp;
  uint32_t* slab;   // n_dst x cap kept sources per row (capped graphs with cap <= FUSE_CAP)
  uint32_t* eslot;  // n_dst x cap: each kept edge's place among its source's edges
  int64_t ncap;
};

// Capped graphs with cap <= FUSE_CAP select their rows in one pass over the
// candidates (k_nbr_select) into a slab of n_dst x cap entries.
bool fused_select(const dsmp_graph_query* q) { return q->cap > 0 && q->cap <= FUSE_CAP; }

GraphWs carve_graph_ws(void* base, const dsmp_graph_query* q, size_t* used) {
  const int64_t n_src = q->n_src, n_dst = q->n_dst;
  Carve c(base);
  GraphWs w;
  w.ncap = 2 * n_src + 64;
  w.part = c.take<float>(BBOX_BLOCKS * 6);
  w.grid = c.take<GridParams>(1);
  w.stats = c.take<GraphStats>(1);
  w.cellid = c.take<uint32_t>(n_src);
  w.ccount = c.take<uint32_t>(w.ncap);
  w.cstart = c.take<int32_t>(w.ncap + 1);
  w.ccur = c.take<uint32_t>(w.ncap);
  w.spos = c.take<float4>(n_src);
  w.sidx = c.take<int32_t>(n_src);
  w.rcnt = c.take<uint32_t>(n_dst);
  w.rraw = c.take<uint32_t>(n_dst);
  w.rowptr_tmp = c.take<int32_t>(n_dst + 1);
  w.indeg = c.take<uint32_t>(n_src);
  w.scur = c.take<uint32_t>(n_src);
  int64_t m = w.ncap > n_src ? w.ncap : n_src;
  w.scan_tmp = c.take<uint32_t>(scan_tmp_elems(m));
  w.slab = fused_select(q) ? c.take<uint32_t>(n_dst * q->cap) : nullptr;
  w.eslot = fused_select(q) ? c.take<uint32_t>(n_dst * q->cap) : nullptr;
  if (used) *used = c.used();
  return w;
}

dsmp_status validate_query(dsmp_handle* h, const dsmp_graph_query* q) {
  DSMP_CHECK(h, q != nullptr, DSMP_INVALID_ARG, "query is NULL");
  DSMP_CHECK(h, q->dim == 2 || q->dim == 3, DSMP_INVALID_ARG, "dim must be 2 or 3");
  DSMP_CHECK(h, q->n_dst >= 0 && q->n_src >= q->n_dst, DSMP_INVALID_ARG, "need 0 <= n_dst <= n_src");
  DSMP_CHECK(h, q->n_src <= INT32_MAX / 2, DSMP_UNSUPPORTED, "n_src too large");
  DSMP_CHECK(h, q->r >= 0.0f && q->r < INFINITY, DSMP_INVALID_ARG, "radius must be finite and >= 0");
  DSMP_CHECK(h, q->cap >= 0, DSMP_INVALID_ARG, "cap must be >= 0");
  DSMP_CHECK(h, q->cap_mode == DSMP_CAP_KNN || q->cap_mode == DSMP_CAP_RANDOM, DSMP_INVALID_ARG,
             "unknown cap mode");
  DSMP_CHECK(h, q->n_src == 0 || q->pos != nullptr, DSMP_INVALID_ARG, "pos is NULL");
  return DSMP_OK;
}

// Phases shared by count and build: grid, cell sort, per-row counts, scan
// into row_ptr.  Then the host reads back E and the largest row.
dsmp_status count_phase(dsmp_handle* h, const dsmp_graph_query* q, const GraphWs& w, int32_t* row_ptr,
                        int64_t* E, uint32_t* maxraw, bool select) {
  const int D = q->dim;
  const float r2 = __builtin_bit_cast(float, 0) + q->r * q->r;   // fl32(r*r)
  hipStream_t s = h->stream;
  int64_t n = q->n_src;
  unsigned nb = n > 0 ? ceil_div(n, 256) : 1;
  if (nb > BBOX_BLOCKS) nb = BBOX_BLOCKS;
  hipLaunchKernelGGL(k_bbox_partial, dim3(nb), dim3(256), 0, s, q->pos, n, D, w.part);
  hipLaunchKernelGGL(k_grid_setup, dim3(1), dim3(64), 0, s, w.part, (int)nb, D, q->r, w.ncap, w.grid,
                     w.stats);
  DSMP_LAUNCHED(h, "grid setup");
  dsmp_status st;
  if ((st = fill_u32(h, w.ccount, w.ncap, 0, w.ccur)) != DSMP_OK) return st;
  // the select pass counts in-degrees (and the scatter's cursors start at zero)
  if (select && (st = fill_u32(h, w.indeg, q->n_src, 0, w.scur)) != DSMP_OK) return st;
  if (n > 0) {
    hipLaunchKernelGGL(k_cell_hash, dim3(ceil_div(n, 256)), dim3(256), 0, s, q->pos, n, D, w.grid,
                       w.cellid, w.ccount);
    DSMP_LAUNCHED(h, "cell hash");
  }
  if ((st = exclusive_scan_u32(h, w.ccount, w.cstart, w.ncap, w.scan_tmp)) != DSMP_OK) return st;
  if (n > 0) {
    hipLaunchKernelGGL(k_cell_scatter, dim3(ceil_div(n, 256)), dim3(256), 0, s, q->pos, n, D,
                       w.cellid, w.cstart, w.ccur, w.spos, w.sidx);
    DSMP_LAUNCHED(h, "cell scatter");
  }
  if (q->n_dst > 0) {
    if (select)
      hipLaunchKernelGGL(k_nbr_select, dim3(ceil_div(q->n_dst, 4)), dim3(256), 0, s, q->pos, q->n_dst,
                         q->n_src, D, r2, q->cap, q->cap_mode, q->seed, w.grid, w.cstart, w.spos, w.sidx,
                         w.rcnt, w.rraw, w.slab, w.indeg, w.eslot);
    else
      hipLaunchKernelGGL(k_nbr_count, dim3(ceil_div(q->n_dst, 4)), dim3(256), 0, s, q->pos, q->n_dst, D,
                         r2, q->cap, w.grid, w.cstart, w.spos, w.sidx, w.rcnt, w.rraw);
    hipLaunchKernelGGL(k_graph_stats, dim3((unsigned)std::min<int64_t>(ceil_div(q->n_dst, 2048), 256)),
                       dim3(256), 0, s, w.rcnt, w.rraw, q->n_dst, w.stats);
    DSMP_LAUNCHED(h, "neighbour count");
  }
  if ((st = exclusive_scan_u32(h, w.rcnt, row_ptr, q->n_dst, w.scan_tmp)) != DSMP_OK) return st;
  GraphStats hs;
  DSMP_HIP(h, hipMemcpyAsync(&hs, w.stats, sizeof(hs), hipMemcpyDeviceToHost, s));
  DSMP_HIP(h, hipStreamSynchronize(s));
  *E = (int64_t)hs.total;
  *maxraw = hs.maxraw;
  DSMP_CHECK(h, hs.maxraw <= (uint32_t)ROW_LIMIT, DSMP_UNSUPPORTED,
             "a destination has %u sources within r (limit %d)", hs.maxraw, ROW_LIMIT);
  DSMP_CHECK(h, *E <= INT32_MAX, DSMP_UNSUPPORTED, "edge count %lld exceeds int32", (long long)*E);
  return DSMP_OK;
}

}  // namespace

extern "C" dsmp_status dsmp_radius_graph_workspace(const dsmp_graph_query* q, size_t* bytes) {
  if (!q || !bytes || q->n_src < 0 || q->n_dst < 0) return DSMP_INVALID_ARG;
  carve_graph_ws(nullptr, q, bytes);
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_radius_graph_count(dsmp_handle* h, const dsmp_graph_query* q, void* ws,
                                               size_t ws_bytes, int64_t* n_edges) {
  if (!h) return DSMP_INVALID_ARG;
  dsmp_status st = validate_query(h, q);
  if (st != DSMP_OK) return st;
  DSMP_CHECK(h, n_edges != nullptr, DSMP_INVALID_ARG, "n_edges is NULL");
  size_t need;
  GraphWs w = carve_graph_ws(ws, q, &need);
  DSMP_CHECK(h, ws != nullptr && ws_bytes >= need, DSMP_WORKSPACE_TOO_SMALL,
             "graph workspace needs %zu bytes", need);
  uint32_t maxraw;
  return count_phase(h, q, w, w.rowptr_tmp, n_edges, &maxraw, false);
}

extern "C" dsmp_status dsmp_radius_graph_build(dsmp_handle* h, const dsmp_graph_query* q, void* ws,
                                               size_t ws_bytes, int64_t edge_capacity, dsmp_graph* g) {
  if (!h) return DSMP_INVALID_ARG;
  dsmp_status st = validate_query(h, q);
  if (st != DSMP_OK) return st;
  DSMP_CHECK(h, g != nullptr && g->row_ptr != nullptr, DSMP_INVALID_ARG, "graph or row_ptr is NULL");
  DSMP_CHECK(h, edge_capacity >= 0, DSMP_INVALID_ARG, "negative edge capacity");
  DSMP_CHECK(h, edge_capacity == 0 || (g->col && g->dst), DSMP_INVALID_ARG, "col or dst is NULL");
  DSMP_CHECK(h, g->csc_ptr != nullptr && (edge_capacity == 0 || g->csc_eid), DSMP_INVALID_ARG,
             "csc arrays are NULL");
  size_t need;
  GraphWs w = carve_graph_ws(ws, q, &need);
  DSMP_CHECK(h, ws != nullptr && ws_bytes >= need, DSMP_WORKSPACE_TOO_SMALL,
             "graph workspace needs %zu bytes", need);
  ProfScope prof(h, DSMP_K_GRAPH);
  int64_t E;
  uint32_t maxraw;
  const bool select = fused_select(q);
  // a symmetric graph (no cap, every source a destination) is its own transpose
  const bool symmetric = q->cap == 0 && q->n_src == q->n_dst;
  st = count_phase(h, q, w, g->row_ptr, &E, &maxraw, select);
  g->n_dst = q->n_dst;
  g->n_src = q->n_src;
  g->n_edges = E;
  if (st != DSMP_OK) return st;
  hipStream_t s = h->stream;
  const float r2 = q->r * q->r;
  // in-degrees start at zero (the count phase zeroed them for the select pass)
  if (!select && !symmetric && (st = fill_u32(h, w.indeg, q->n_src, 0, w.scur)) != DSMP_OK) return st;
  // When every row fit the select pass, the in-degrees are complete and the
  // transpose is placed with the rows; otherwise the fill kernel builds the
  // larger rows and the transpose is scattered from col afterwards.
  const bool overflow = select && maxraw > (uint32_t)FUSE_LIM;
  const bool place_csc = select && !overflow;
  if (place_csc && (st = exclusive_scan_u32(h, w.indeg, g->csc_ptr, q->n_src, w.scan_tmp)) != DSMP_OK)
    return st;
  if (select && q->n_dst > 0 && E > 0) {
    const int64_t nslab = q->n_dst * q->cap;
    hipLaunchKernelGGL(k_nbr_place, dim3((unsigned)ceil_div(nslab, 256)), dim3(256), 0, s, q->n_dst,
                       q->cap, w.rraw, g->row_ptr, w.slab, w.eslot, place_csc ? g->csc_ptr : nullptr,
                       edge_capacity, g->col, g->dst, g->csc_eid);
    DSMP_LAUNCHED(h, "neighbour place");
  }
  // every row without the fused select, or with more candidates than it holds
  if (q->n_dst > 0 && E > 0 && (!select || overflow)) {
    int lim = 64;
    while (lim < (int)maxraw) lim <<= 1;
    // up to four rows per block within 48 KB of shared memory (lim <= 4096)
    const int rows = std::min(4, std::max(1, 49152 / (lim * 12)));
    const size_t lds = (size_t)rows * lim * 12;
    hipLaunchKernelGGL(k_nbr_fill, dim3((unsigned)ceil_div(q->n_dst, rows)), dim3(64 * rows), lds, s,
                       q->pos, q->n_dst,
                       q->n_src, q->dim, r2, q->cap, q->cap_mode, q->seed, lim, w.grid, w.cstart,
                       w.spos, w.sidx, g->row_ptr, edge_capacity, g->col, g->dst,
                       symmetric ? nullptr : w.indeg, select ? w.rraw : nullptr, FUSE_LIM);
    DSMP_LAUNCHED(h, "neighbour fill");
  }
  DSMP_CHECK(h, E <= edge_capacity, DSMP_CAPACITY, "graph has %lld edges, capacity %lld",
             (long long)E, (long long)edge_capacity);
  if (symmetric) {
    const int64_t n_ptr = q->n_dst + 1;
    hipLaunchKernelGGL(k_csc_symmetric, dim3((unsigned)ceil_div(std::max<int64_t>(E, n_ptr), 256)), dim3(256), 0, s,
                       g->row_ptr, n_ptr, g->col, g->dst, E, g->csc_ptr, g->csc_eid);
    DSMP_LAUNCHED(h, "csc (symmetric graph)");
    return DSMP_OK;
  }
  if (!place_csc && (st = exclusive_scan_u32(h, w.indeg, g->csc_ptr, q->n_src, w.scan_tmp)) != DSMP_OK)
    return st;
  if (E > 0) {
    if (!place_csc)
      hipLaunchKernelGGL(k_csc_scatter, dim3(ceil_div(E, 256)), dim3(256), 0, s, g->col, E, g->csc_ptr,
                         w.scur, g->csc_eid);
    hipLaunchKernelGGL(k_csc_sort, dim3((unsigned)ceil_div(q->n_src, 4 * CSC_COLS)), dim3(256), 0, s,
                       g->csc_ptr, q->n_src, g->csc_eid);
    DSMP_LAUNCHED(h, "csc build");
  }
  return DSMP_OK;
}
