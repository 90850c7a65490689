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

// One thread: reduce the partial boxes and choose the cell size.  Cells are
// at least r*(1 + 2^-10) wide, so two points that pass the float32 radius
// test always sit in the same or adjacent cells (cell coordinates are formed
// in double, see cell_coord); the grid is coarsened by doubling until it has
// at most `cap` cells.
__global__ void k_grid_setup(const float* __restrict__ part, int nb, int D, float r, int64_t cap,
                             GridParams* __restrict__ g, GraphStats* __restrict__ st) {
  if (threadIdx.x != 0) return;
  float lo[3] = {INFINITY, INFINITY, INFINITY}, hi[3] = {-INFINITY, -INFINITY, -INFINITY};
  for (int b = 0; b < nb; ++b)
    for (int a = 0; a < 3; ++a) {
      lo[a] = fminf(lo[a], part[b * 6 + a]);
      hi[a] = fmaxf(hi[a], part[b * 6 + 3 + a]);
    }
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

// Visit the candidate ranges of destination i: for every neighbouring cell
// row (3 in 2-D, 9 in 3-D) the three cells along x are one contiguous range of
// the cell-sorted arrays.
template <typename F>
__device__ __forceinline__ void for_each_candidate_range(float3 p, int D, const GridParams& g,
                                                         const int32_t* __restrict__ cstart, F f) {
  int cx = cell_coord(p.x, g.lo[0], g.inv_c, g.dims[0]);
  int cy = cell_coord(p.y, g.lo[1], g.inv_c, g.dims[1]);
  int cz = D == 3 ? cell_coord(p.z, g.lo[2], g.inv_c, g.dims[2]) : 0;
  int x0 = cx > 0 ? cx - 1 : 0, x1 = cx + 1 < g.dims[0] ? cx + 1 : g.dims[0] - 1;
  int zlo = D == 3 ? -1 : 0, zhi = D == 3 ? 1 : 0;
  for (int dz = zlo; dz <= zhi; ++dz) {
    int z = cz + dz;
    if (z < 0 || z >= g.dims[2]) continue;
    for (int dy = -1; dy <= 1; ++dy) {
      int y = cy + dy;
      if (y < 0 || y >= g.dims[1]) continue;
      int base = g.dims[0] * (y + g.dims[1] * z);
      f(cstart[base + x0], cstart[base + x1 + 1]);
    }
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
  uint32_t cnt = 0;
  for_each_candidate_range(pi, D, g, cstart, [&](int a, int b) {
    for (int t = a + lane; t < b; t += 64) {
      float4 q = spos[t];
      float d2 = dist2(pi, make_float3(q.x, q.y, q.z), D);
      if (d2 <= r2 && sidx[t] != (int32_t)i) ++cnt;
    }
  });
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
  if (lane == 0) {
    rcnt[i] = (cap > 0 && cnt > (uint32_t)cap) ? (uint32_t)cap : cnt;
    rraw[i] = cnt;
  }
}

// Edge total (64-bit) and largest pre-cap row count, one block.
__global__ __launch_bounds__(1024) void k_graph_stats(const uint32_t* __restrict__ rcnt,
                                                      const uint32_t* __restrict__ rraw, int64_t n_dst,
                                                      GraphStats* __restrict__ st) {
  __shared__ unsigned long long ssum[1024];
  __shared__ uint32_t smax[1024];
  unsigned long long s = 0;
  uint32_t m = 0;
  for (int64_t i = threadIdx.x; i < n_dst; i += 1024) {
    s += rcnt[i];
    m = rraw[i] > m ? rraw[i] : m;
  }
  ssum[threadIdx.x] = s;
  smax[threadIdx.x] = m;
  __syncthreads();
  for (int o = 512; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) {
      ssum[threadIdx.x] += ssum[threadIdx.x + o];
      smax[threadIdx.x] = smax[threadIdx.x + o] > smax[threadIdx.x] ? smax[threadIdx.x + o] : smax[threadIdx.x];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    st->total = ssum[0];
    st->maxraw = smax[0];
  }
}

// Bitonic sort of P (power of two) 64-bit keys with 32-bit payload, by one
// wave (the block is one wave, so __syncthreads is a wave barrier).
__device__ void bitonic_kv(uint64_t* key, int32_t* val, int P) {
  for (int k = 2; k <= P; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int t = threadIdx.x; t < P; t += 64) {
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
      __syncthreads();
    }
}

__device__ void bitonic_u32(uint32_t* key, int P) {
  for (int k = 2; k <= P; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int t = threadIdx.x; t < P; t += 64) {
        int u = t ^ j;
        if (u > t) {
          bool up = (t & k) == 0;
          uint32_t a = key[t], b = key[u];
          if ((a > b) == up) { key[t] = b; key[u] = a; }
        }
      }
      __syncthreads();
    }
}

__device__ __forceinline__ int next_pow2(int n) {
  int p = 1;
  while (p < n) p <<= 1;
  return p;
}

// One wave per destination row: gather the sources that pass the test into
// LDS, apply the cap by sorting on (d2, j) or on the hashed key, sort the kept
// sources by index and write the row.
__global__ __launch_bounds__(64) void k_nbr_fill(const float* __restrict__ pos, int64_t n_dst,
                                                 int64_t n_src, int D, float r2, int cap,
                                                 int cap_mode, uint64_t seed, int lim,
                                                 const GridParams* __restrict__ gp,
                                                 const int32_t* __restrict__ cstart,
                                                 const float4* __restrict__ spos,
                                                 const int32_t* __restrict__ sidx,
                                                 const int32_t* __restrict__ row_ptr,
                                                 int64_t capacity, int32_t* __restrict__ col,
                                                 int32_t* __restrict__ dst) {
  extern __shared__ __align__(16) unsigned char smem[];
  uint64_t* key = reinterpret_cast<uint64_t*>(smem);
  int32_t* val = reinterpret_cast<int32_t*>(smem + (size_t)lim * 8);
  const int lane = threadIdx.x;
  const int64_t i = blockIdx.x;
  if (i >= n_dst) return;
  const GridParams g = *gp;
  const float3 pi = load_pos(pos, i, D);
  int n = 0;
  for_each_candidate_range(pi, D, g, cstart, [&](int a, int b) {
    for (int t0 = a; t0 < b; t0 += 64) {
      int t = t0 + lane;
      bool pass = false;
      float d2 = 0.0f;
      int32_t j = -1;
      if (t < b) {
        float4 q = spos[t];
        d2 = dist2(pi, make_float3(q.x, q.y, q.z), D);
        j = sidx[t];
        pass = d2 <= r2 && j != (int32_t)i;
      }
      uint64_t m = __ballot(pass);
      if (pass) {
        int slot = n + __popcll(m & ((1ull << lane) - 1ull));
        uint64_t k = cap_mode == DSMP_CAP_KNN
                         ? (((uint64_t)__float_as_uint(d2)) << 32) | (uint32_t)j
                         : splitmix64(seed, (uint64_t)i * (uint64_t)n_src + (uint64_t)j);
        key[slot] = k;
        val[slot] = j;
      }
      n += __popcll(m);
    }
  });
  __syncthreads();
  if (cap > 0 && n > cap) {
    int P = next_pow2(n);
    for (int t = n + lane; t < P; t += 64) { key[t] = ~0ull; val[t] = INT32_MAX; }
    __syncthreads();
    bitonic_kv(key, val, P);
    n = cap;
  }
  // sort the kept sources by index (reuse the key array as uint32 scratch)
  uint32_t* js = reinterpret_cast<uint32_t*>(key);
  for (int t = lane; t < n; t += 64) js[t] = (uint32_t)val[t];
  __syncthreads();
  int P = next_pow2(n > 0 ? n : 1);
  for (int t = n + lane; t < P; t += 64) js[t] = 0xFFFFFFFFu;
  __syncthreads();
  bitonic_u32(js, P);
  const int64_t base = row_ptr[i];
  for (int t = lane; t < n; t += 64) {
    int64_t e = base + t;
    if (e < capacity) {
      col[e] = (int32_t)js[t];
      dst[e] = (int32_t)i;
    }
  }
}

__global__ __launch_bounds__(256) void k_csc_count(const int32_t* __restrict__ col, int64_t E,
                                                   uint32_t* __restrict__ indeg) {
  int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < E) atomicAdd(&indeg[col[e]], 1u);
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
__global__ __launch_bounds__(64) void k_csc_sort(const int32_t* __restrict__ csc_ptr, int64_t n_src,
                                                 int32_t* __restrict__ csc_eid) {
  __shared__ uint32_t buf[CSC_SORT_LDS];
  const int64_t j = blockIdx.x;
  if (j >= n_src) return;
  const int a = csc_ptr[j], b = csc_ptr[j + 1], n = b - a;
  if (n <= 1) return;
  if (n <= CSC_SORT_LDS) {
    int P = next_pow2(n);
    for (int t = threadIdx.x; t < P; t += 64) buf[t] = t < n ? (uint32_t)csc_eid[a + t] : 0xFFFFFFFFu;
    __syncthreads();
    bitonic_u32(buf, P);
    for (int t = threadIdx.x; t < n; t += 64) csc_eid[a + t] = (int32_t)buf[t];
  } else if (threadIdx.x == 0) {
    for (int t = a + 1; t < b; ++t) {
      int32_t v = csc_eid[t];
      int u = t - 1;
      while (u >= a && csc_eid[u] > v) { csc_eid[u + 1] = csc_eid[u]; --u; }
      csc_eid[u + 1] = v;
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
  int64_t ncap;
};

GraphWs carve_graph_ws(void* base, int64_t n_src, int64_t n_dst, size_t* used) {
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
                        int64_t* E, uint32_t* maxraw) {
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
    hipLaunchKernelGGL(k_nbr_count, dim3(ceil_div(q->n_dst, 4)), dim3(256), 0, s, q->pos, q->n_dst, D,
                       r2, q->cap, w.grid, w.cstart, w.spos, w.sidx, w.rcnt, w.rraw);
    hipLaunchKernelGGL(k_graph_stats, dim3(1), dim3(1024), 0, s, w.rcnt, w.rraw, q->n_dst, w.stats);
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
  carve_graph_ws(nullptr, q->n_src, q->n_dst, bytes);
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_radius_graph_count(dsmp_handle* h, const dsmp_graph_query* q, void* ws,
                                               size_t ws_bytes, int64_t* n_edges) {
  if (!h) return DSMP_INVALID_ARG;
  dsmp_status st = validate_query(h, q);
  if (st != DSMP_OK) return st;
  DSMP_CHECK(h, n_edges != nullptr, DSMP_INVALID_ARG, "n_edges is NULL");
  size_t need;
  GraphWs w = carve_graph_ws(ws, q->n_src, q->n_dst, &need);
  DSMP_CHECK(h, ws != nullptr && ws_bytes >= need, DSMP_WORKSPACE_TOO_SMALL,
             "graph workspace needs %zu bytes", need);
  uint32_t maxraw;
  return count_phase(h, q, w, w.rowptr_tmp, n_edges, &maxraw);
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
  GraphWs w = carve_graph_ws(ws, q->n_src, q->n_dst, &need);
  DSMP_CHECK(h, ws != nullptr && ws_bytes >= need, DSMP_WORKSPACE_TOO_SMALL,
             "graph workspace needs %zu bytes", need);
  ProfScope prof(h, DSMP_K_GRAPH);
  int64_t E;
  uint32_t maxraw;
  st = count_phase(h, q, w, g->row_ptr, &E, &maxraw);
  g->n_dst = q->n_dst;
  g->n_src = q->n_src;
  g->n_edges = E;
  if (st != DSMP_OK) return st;
  hipStream_t s = h->stream;
  const float r2 = q->r * q->r;
  if (q->n_dst > 0 && E > 0) {
    int lim = 64;
    while (lim < (int)maxraw) lim <<= 1;
    size_t lds = (size_t)lim * 12;
    hipLaunchKernelGGL(k_nbr_fill, dim3((unsigned)q->n_dst), dim3(64), lds, s, q->pos, q->n_dst,
                       q->n_src, q->dim, r2, q->cap, q->cap_mode, q->seed, lim, w.grid, w.cstart,
                       w.spos, w.sidx, g->row_ptr, edge_capacity, g->col, g->dst);
    DSMP_LAUNCHED(h, "neighbour fill");
  }
  DSMP_CHECK(h, E <= edge_capacity, DSMP_CAPACITY, "graph has %lld edges, capacity %lld",
             (long long)E, (long long)edge_capacity);
  if (q->cap == 0 && q->n_src == q->n_dst) {
    // symmetric graph: the transpose is the row structure itself
    const int64_t n_ptr = q->n_dst + 1;
    hipLaunchKernelGGL(k_csc_symmetric, dim3((unsigned)ceil_div(std::max<int64_t>(E, n_ptr), 256)), dim3(256), 0, s,
                       g->row_ptr, n_ptr, g->col, g->dst, E, g->csc_ptr, g->csc_eid);
    DSMP_LAUNCHED(h, "csc (symmetric graph)");
    return DSMP_OK;
  }
  if ((st = fill_u32(h, w.indeg, q->n_src, 0, w.scur)) != DSMP_OK) return st;
  if (E > 0) {
    hipLaunchKernelGGL(k_csc_count, dim3(ceil_div(E, 256)), dim3(256), 0, s, g->col, E, w.indeg);
    DSMP_LAUNCHED(h, "csc count");
  }
  if ((st = exclusive_scan_u32(h, w.indeg, g->csc_ptr, q->n_src, w.scan_tmp)) != DSMP_OK) return st;
  if (E > 0) {
    hipLaunchKernelGGL(k_csc_scatter, dim3(ceil_div(E, 256)), dim3(256), 0, s, g->col, E, g->csc_ptr,
                       w.scur, g->csc_eid);
    hipLaunchKernelGGL(k_csc_sort, dim3((unsigned)q->n_src), dim3(64), 0, s, g->csc_ptr, q->n_src,
                       g->csc_eid);
    DSMP_LAUNCHED(h, "csc build");
  }
  return DSMP_OK;
}
