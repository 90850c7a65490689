// NNConv layer forward (eq. (1), eq. (ii); Algorithm 1, graph-convolution step
// with the residual hop update), parameter packing, and the edge contraction
// that the backward pass reuses for the feature gradient.
//
// Edge contraction.  For edge e = (i <- j) the message is
//     m_e[q] = sum_p h_j[p] * ( sum_k W3[p*d+q][k] z_e[k] + b3[p*d+q] ).
// The d x d kernel matrix is never formed.  For each p the 32-row blocks of
// W3[p*d + q][:] (rows q) are the A operand of a bf16 (or fp32) MFMA chain
// over k, the edge tile's z vectors (held in registers for the whole loop)
// are the B operand, and the 32x32 product is scaled by h_j[p] (one value per
// lane: the lane's column is its edge) and accumulated.  The b3 term is one
// more small MFMA product, B3^T h_j, that initialises the accumulators.  W3
// is streamed through LDS in double-buffered chunks shared by the four waves
// of a workgroup, and each A fragment feeds two edge tiles.
//
// Segmented mean without atomics: the edges of a workgroup tile are sorted by
// destination, so the tile's messages go to LDS and one thread per
// (destination, column) sums its run in edge order.  Destinations that start
// or end outside the tile leave a partial sum (first and last run of every
// tile); the node kernel adds those partials in tile order.
#include "nnconv.hpp"


using namespace dsmp;

namespace {

template <typename T>
__device__ __forceinline__ void set_el(typename MT<T>::frag& f, int i, float v);
template <>
__device__ __forceinline__ void set_el<__bf16>(bf16x8& f, int i, float v) { f[i] = (__bf16)v; }
template <>
__device__ __forceinline__ void set_el<float>(float& f, int, float v) { f = v; }

template <typename T>
__device__ __forceinline__ typename MT<T>::frag ld_frag(const void* p) {
  return *reinterpret_cast<const typename MT<T>::frag*>(p);
}

template <typename T>
__device__ __forceinline__ typename MT<T>::frag zero_frag() {
  typename MT<T>::frag f;
  if constexpr (sizeof(f) == 4) f = 0.0f;
  else for (int i = 0; i < 8; ++i) f[i] = (__bf16)0.0f;
  return f;
}

__device__ __forceinline__ float to_f(__bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f(float x) { return x; }

template <typename T, int DL, int H1, int H2>
struct Shape {
  static constexpr int KS = MT<T>::KS, EPL = MT<T>::EPL, NT = 2, TILE = EDGE_TILE;
  static constexpr int QT = DL / 32, KT = H2 / 32;
  static constexpr int SK1 = H1 / KS, SK2 = H2 / KS, SKD = DL / KS;
  static constexpr int ESZ = sizeof(T);
  static constexpr int ROWB = H2 * ESZ + 16;
  static constexpr int RCH = (DL * H2 * ESZ <= 32768) ? DL : (32768 / (H2 * ESZ));
  static constexpr int CPP = DL / RCH, QPC = RCH / 32, NCH = DL * CPP;
  static constexpr int STAGE = RCH * ROWB;
  static constexpr int HROWB = DL * ESZ + 16;
  static constexpr int MSGW = DL + 4;
  // The scaling of a q-block's products is deferred past the next block's
  // MFMA chain when the extra accumulator set fits the register budget.
  static constexpr bool PIPE = DL <= 64;
  static constexpr int AD = 4;   // A-fragment read depth of the main loop
  // W2 staged in the two W3 buffers, in pieces of W2R rows when it is larger
  static constexpr int W2B = H1 * ESZ + 16;
  static constexpr int W2R_FIT = (2 * STAGE / W2B) / 32 * 32;
  static constexpr int W2R = W2R_FIT < H2 ? W2R_FIT : H2, NW2 = H2 / W2R;
  static_assert(W2R >= 32 && H2 % W2R == 0, "W2 pieces");
  static constexpr int W1BYTES = H1 * 8 * 4 + H1 * 4;   // W1 [2][H1/2][8], b1 [2][H1/2] (fp32)
  static constexpr int LDS_MAIN = 2 * STAGE + TILE * HROWB + W1BYTES;
  static constexpr int LDS_MSG = TILE * MSGW * 4;
  static constexpr int LDS = LDS_MAIN > LDS_MSG ? LDS_MAIN : LDS_MSG;
};


// Two workgroups per CU when registers and LDS allow (d <= 64), so one
// workgroup's MFMA chains overlap the other's barriers and epilogues.
template <typename T, int DL, int H1, int H2, int MODE>
__global__ __launch_bounds__(256, (DL <= 64 && H2 * sizeof(T) <= 256) ? 2 : 1) void k_edge_contract(EdgeArgs a) {
  using S = Shape<T, DL, H1, H2>;
  using M = MT<T>;
  using frag = typename M::frag;
  constexpr int KS = S::KS, EPL = S::EPL, NT = S::NT, TILE = S::TILE, ESZ = S::ESZ;
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* stage0 = smem;
  unsigned char* htile = smem + 2 * S::STAGE;
  float* w1s = reinterpret_cast<float*>(htile + TILE * S::HROWB);
  float* msg = reinterpret_cast<float*>(smem);

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  const int64_t tile = blockIdx.x, t0 = tile * TILE;
  const int64_t tend = t0 + TILE < a.E ? t0 + TILE : a.E;
  const unsigned char* P = a.packed;
  const unsigned char* A3 = P + (MODE == MODE_FWD ? a.L.w3f : a.L.w3q);
  using St = LdsStage<S::RCH, H2 * ESZ>;
  static_assert(St::BYTES == S::STAGE, "stage layout");
  auto chunk = [&](int c) {
    return A3 + ((size_t)(c / S::CPP) * DL + (size_t)(c % S::CPP) * S::RCH) * H2 * ESZ;
  };
  St stg;
  stg.init();

  // Direct-to-LDS loads go out first so their latency overlaps the id and
  // attribute loads: the tile's gathered rows (h_j in the forward, g_i for
  // the feature gradient; rows past E take row 0 and are never read back),
  // then the first-layer weights and W2 (forward) or the first W3 chunk.
  // The kernel-MLP-only form (z and z1 for the aggregate form) stops after z.
  if constexpr (MODE != MODE_MLP) {
    constexpr int HU = DL * ESZ / 16, PITCH = HU + 1, UNITS = TILE * PITCH;
    const int wbase = tid & ~63;
#pragma unroll
    for (int i = 0; i < (UNITS + 255) / 256; ++i) {
      const int U = i * 256 + tid;
      if (UNITS % 256 == 0 || U < UNITS) {
        const int r = U / PITCH, c = U % PITCH;
        const int64_t s = t0 + r;
        int node = 0;
        if (s < a.E) node = MODE == MODE_FWD ? a.col[s] : a.dst[a.csc_eid[s]];
        __builtin_amdgcn_global_load_lds(
            (gbl_void_t*)(a.gath + (size_t)node * DL * ESZ + (c < HU ? c : 0) * 16),
            (lds_void_t*)(htile + (size_t)(i * 256 + wbase) * 16), 16, 0, 0);
      }
    }
  }
  if constexpr (MODE != MODE_DH) {
    lds_copy_async(P + a.L.w1l, reinterpret_cast<unsigned char*>(w1s), H1 * 8 * 4 / 16);
    lds_copy_async(P + a.L.b1l, reinterpret_cast<unsigned char*>(w1s + H1 * 8), H1 * 4 / 16);
    LdsStage<S::W2R, H1 * ESZ> w2st;
    w2st.init();
    w2st.issue(P + a.L.w2p, stage0);
  } else {
    stg.issue(chunk(0), stage0);
  }

  int64_t eid[NT];
  int dnode[NT], snode[NT], hrow[NT];
  bool valid[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    hrow[t] = (wv * NT + t) * 32 + l32;
    int64_t s = t0 + hrow[t];
    valid[t] = s < a.E;
    int64_t e = valid[t] ? (MODE != MODE_DH ? s : (int64_t)a.csc_eid[s]) : 0;
    eid[t] = e;
    dnode[t] = valid[t] ? a.dst[e] : 0;
    snode[t] = valid[t] ? a.col[e] : 0;
  }

  // B operand of the contraction: z_e, in the permuted register order
  frag zB[NT][S::SK2];
  if constexpr (MODE != MODE_DH) {
    float x[NT][8];
#pragma unroll
    for (int t = 0; t < NT; ++t) edge_attr(a.node_attr, a.dim, a.attr_mode, dnode[t], snode[t], x[t]);
    if constexpr (sizeof(T) == 2) {
      if (a.xE) {   // for the backward: bf16 high parts (lane half 0), then low parts (half 1)
#pragma unroll
        for (int t = 0; t < NT; ++t)
          if (valid[t]) {
            float v[8];
#pragma unroll
            for (int c = 0; c < 8; ++c) {
              const float hi = (float)(__bf16)x[t][c];
              v[c] = hh ? x[t][c] - hi : hi;
            }
            *reinterpret_cast<bf16x8*>(a.xE + (size_t)eid[t] * 32 + hh * 16) = pack_frag<__bf16>(v);
          }
      }
    }
    stage_wait();
    __syncthreads();   // rows, W1 and W2 are in LDS
    frag z1B[NT][S::SK1];
    // ReLU masks for the backward: bit s*EPL+u of the lane's half is
    // [value at position s*KS + hh*EPL + u > 0] (z1 words, then z words)
    constexpr int MW1 = H1 / 64, MW2 = H2 / 64;
    uint32_t m1[NT][MW1], m2[NT][MW2];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
      for (int w = 0; w < MW1; ++w) m1[t][w] = 0u;
#pragma unroll
      for (int w = 0; w < MW2; ++w) m2[t][w] = 0u;
    }
    const float* w1h = w1s + hh * (H1 / 2) * 8;
    const float* b1h = w1s + H1 * 8 + hh * (H1 / 2);
#pragma unroll
    for (int s = 0; s < S::SK1; ++s) {
      float zv[NT][EPL];
#pragma unroll
      for (int u = 0; u < EPL; ++u) {
        const int n = s * EPL + u;
        const float bn = b1h[n];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const float v = layer1_pre(w1h + n * 8, bn, x[t]);
          zv[t][u] = relu_mask(v, m1[t][n / 32], n % 32);
        }
      }
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        z1B[t][s] = pack_frag<T>(zv[t]);
        // fold the bits into their words here rather than at the store
#pragma unroll
        for (int w = 0; w < MW1; ++w) asm("" : "+v"(m1[t][w]));
      }
    }
    if (a.z1E) {
#pragma unroll
      for (int t = 0; t < NT; ++t)
        if (valid[t])
#pragma unroll
          for (int s = 0; s < S::SK1; ++s)
            *reinterpret_cast<frag*>(a.z1E + ((size_t)eid[t] * H1 + s * KS + hh * EPL) * ESZ) = z1B[t][s];
    }
    const float* b2 = reinterpret_cast<const float*>(P + a.L.b2);
#pragma unroll
    for (int piece = 0; piece < S::NW2; ++piece) {
      if (piece > 0) {
        __syncthreads();   // every wave is done with the previous piece
        LdsStage<S::W2R, H1 * ESZ> w2st;
        w2st.init();
        w2st.issue(P + a.L.w2p + (size_t)piece * S::W2R * H1 * ESZ, stage0);
        stage_wait();
        __syncthreads();
      }
#pragma unroll
      for (int kl = 0; kl < S::W2R / 32; ++kl) {
        const int kt = piece * (S::W2R / 32) + kl;
        f32x16 C[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) C[t] = f32x16{};
#pragma unroll
        for (int s = 0; s < S::SK1; ++s) {
          frag A = ld_frag<T>(stage0 + (kl * 32 + l32) * S::W2B + (s * KS + hh * EPL) * ESZ);
#pragma unroll
          for (int t = 0; t < NT; ++t) C[t] = M::mma(A, z1B[t][s], C[t]);
        }
        float bb[16];
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4) {
          f32x4 v = *reinterpret_cast<const f32x4*>(b2 + kt * 32 + 8 * a4 + 4 * hh);
          bb[4 * a4] = v[0]; bb[4 * a4 + 1] = v[1]; bb[4 * a4 + 2] = v[2]; bb[4 * a4 + 3] = v[3];
        }
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int i0 = 0; i0 < 16; i0 += EPL) {
            float zv[EPL];
#pragma unroll
            for (int u = 0; u < EPL; ++u) {
              const float v = C[t][i0 + u] + bb[i0 + u];
              const int b = 16 * kt + i0 + u;
              zv[u] = relu_mask(v, m2[t][b / 32], b % 32);
            }
            zB[t][(16 * kt + i0) / EPL] = pack_frag<T>(zv);
          }
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int w = 0; w < MW2; ++w) asm("" : "+v"(m2[t][w]));
      }
    }
    if (a.zE) {
#pragma unroll
      for (int t = 0; t < NT; ++t)
        if (valid[t])
#pragma unroll
          for (int s = 0; s < S::SK2; ++s)
            *reinterpret_cast<frag*>(a.zE + ((size_t)eid[t] * H2 + s * KS + hh * EPL) * ESZ) = zB[t][s];
    }
    if (a.zmask) {
#pragma unroll
      for (int t = 0; t < NT; ++t)
        if (valid[t]) {
          uint32_t* mb = reinterpret_cast<uint32_t*>(a.zmask + (size_t)eid[t] * ((H1 + H2) / 8));
#pragma unroll
          for (int w = 0; w < MW1; ++w) mb[hh * MW1 + w] = m1[t][w];
#pragma unroll
          for (int w = 0; w < MW2; ++w) mb[2 * MW1 + hh * MW2 + w] = m2[t][w];
        }
    }
    if constexpr (MODE == MODE_MLP) return;
    __syncthreads();   // every wave is done with W2: the first W3 chunk takes its place
    stg.issue(chunk(0), stage0);
  } else {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int s = 0; s < S::SK2; ++s)
        zB[t][s] = valid[t] ? ld_frag<T>(a.zE + ((size_t)eid[t] * H2 + s * KS + hh * EPL) * ESZ)
                            : zero_frag<T>();
    stage_wait();
    __syncthreads();   // gathered rows (and the first W3 chunk) are in LDS
  }

  // accumulators start at the bias term  B3^T u  (u = gathered row)
  f32x16 acc[NT][S::QT];
  {
    const unsigned char* bop = P + (MODE == MODE_FWD ? a.L.b3t : a.L.b3n);
#pragma unroll
    for (int qt = 0; qt < S::QT; ++qt) {
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[t][qt] = f32x16{};
#pragma unroll
      for (int ps = 0; ps < S::SKD; ++ps) {
        frag A = ld_frag<T>(bop + ((size_t)(qt * 32 + l32) * DL + ps * KS + hh * EPL) * ESZ);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          frag B = ld_frag<T>(htile + hrow[t] * S::HROWB + (ps * KS + hh * EPL) * ESZ);
          acc[t][qt] = M::mma(A, B, acc[t][qt]);
        }
      }
    }
  }
  if constexpr (MODE == MODE_FWD) {
    stage_wait();
    __syncthreads();   // first W3 chunk is in LDS
  }

  // main loop over p: W3 rows (p*d + q), chunks of RCH rows, double-buffered
  // in LDS and fetched one chunk ahead straight into LDS.  The products of
  // one q-block are scaled into the accumulators after the next block's MFMA
  // chain has been issued, so the scaling overlaps the matrix work.
  f32x16 Cp[NT];
  float scp[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    Cp[t] = f32x16{};
    scp[t] = 0.0f;
  }
  for (int p = 0; p < DL; ++p) {
    float sc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
      sc[t] = to_f(*reinterpret_cast<const T*>(htile + hrow[t] * S::HROWB + p * ESZ));
#pragma unroll
    for (int cc = 0; cc < S::CPP; ++cc) {
      const int c = p * S::CPP + cc;
      const int buf = c & 1;
      if (c + 1 < S::NCH) stg.issue(chunk(c + 1), stage0 + (buf ^ 1) * S::STAGE);
      const unsigned char* sb = stage0 + buf * S::STAGE;
      // A fragments of the chunk, read AD-1 steps ahead of their products
      constexpr int NS = S::QPC * S::SK2, AD = S::AD;
      auto a_at = [&](int j) {
        return sb + ((j / S::SK2) * 32 + l32) * S::ROWB + ((j % S::SK2) * KS + hh * EPL) * ESZ;
      };
      frag Ab[AD];
#pragma unroll
      for (int j = 0; j < AD - 1; ++j) Ab[j] = ld_frag<T>(a_at(j));
#pragma unroll
      for (int qq = 0; qq < S::QPC; ++qq) {
        f32x16 C[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) C[t] = f32x16{};
        // retire the previous q-block (block QT-1 of the previous p before
        // block 0) a few registers per step, between this block's products
        const int prev = (cc * S::QPC + qq + S::QT - 1) % S::QT;
#pragma unroll
        for (int s = 0; s < S::SK2; ++s) {
          const int j = qq * S::SK2 + s;
          if (j + AD - 1 < NS) Ab[(j + AD - 1) % AD] = ld_frag<T>(a_at(j + AD - 1));
#pragma unroll
          for (int t = 0; t < NT; ++t) C[t] = M::mma(Ab[j % AD], zB[t][s], C[t]);
          if constexpr (S::PIPE) {
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
              for (int pq = 0; pq < S::QT; ++pq)
                if (pq == prev)
#pragma unroll
                  for (int r = s * 16 / S::SK2; r < (s + 1) * 16 / S::SK2; ++r) acc[t][pq][r] += scp[t] * Cp[t][r];
          }
          // keep the read-ahead and the interleaving in this order
          __builtin_amdgcn_sched_barrier(0);
        }
        if constexpr (S::PIPE) {
#pragma unroll
          for (int t = 0; t < NT; ++t) {
            Cp[t] = C[t];
            scp[t] = sc[t];
          }
        } else {
#pragma unroll
          for (int t = 0; t < NT; ++t) acc[t][cc * S::QPC + qq] += sc[t] * C[t];
        }
      }
      stage_wait();
      __syncthreads();
    }
  }
  if constexpr (S::PIPE) {
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t][S::QT - 1] += scp[t] * Cp[t];
  }

  // messages to LDS, then per-destination (or per-source) runs
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int qt = 0; qt < S::QT; ++qt)
#pragma unroll
      for (int a4 = 0; a4 < 4; ++a4) {
        f32x4 v = {acc[t][qt][4 * a4], acc[t][qt][4 * a4 + 1], acc[t][qt][4 * a4 + 2],
                   acc[t][qt][4 * a4 + 3]};
        *reinterpret_cast<f32x4*>(msg + hrow[t] * S::MSGW + qt * 32 + 8 * a4 + 4 * hh) = v;
      }
  __syncthreads();
  const int32_t* ptr = MODE == MODE_FWD ? a.row_ptr : a.csc_ptr;
  const int64_t i_first = MODE == MODE_FWD ? a.dst[t0] : a.col[a.csc_eid[t0]];
  const int64_t i_last = MODE == MODE_FWD ? a.dst[tend - 1] : a.col[a.csc_eid[tend - 1]];
  constexpr int G = 256 / DL;
  const int q = tid % DL;
  for (int64_t i = i_first + tid / DL; i <= i_last; i += G) {
    const int64_t pa = ptr[i], pb = ptr[i + 1];
    const int64_t lo = pa > t0 ? pa : t0, hi = pb < tend ? pb : tend;
    if (lo >= hi) continue;
    float s = 0.0f;
    for (int64_t u = lo; u < hi; ++u) s += msg[(u - t0) * S::MSGW + q];
    if (pa >= t0 && pb <= tend) a.out_direct[i * DL + q] = s;
    else a.out_part[(tile * 2 + (pa < t0 ? 0 : 1)) * DL + q] = s;
  }
}

// Sum of the run of segment i at column q from the tile sums the edge kernel
// left: one direct value when the run sits in one tile, else the partials of
// the tiles it crosses, in tile order.
__device__ __forceinline__ float segment_sum(const int32_t* __restrict__ ptr, int64_t i, int q, int DL,
                                             const float* __restrict__ direct,
                                             const float* __restrict__ part) {
  const int64_t pa = ptr[i], pb = ptr[i + 1];
  if (pb <= pa) return 0.0f;
  const int64_t ta = pa / EDGE_TILE, tb = (pb - 1) / EDGE_TILE;
  if (ta == tb) return direct[i * DL + q];
  float s = part[(ta * 2 + 1) * DL + q];
  for (int64_t t = ta + 1; t < tb; ++t) s += part[(t * 2) * DL + q];
  s += part[(tb * 2) * DL + q];
  return s;
}

struct NodeArgs {
  int64_t n_dst;
  const int32_t* row_ptr;
  const unsigned char* h_in;   // [n_src][d] layer dtype
  const float* direct;
  const float* part;
  const float* wr;             // [d][d] fp32
  const float* br;             // [d]
  float* h_out;
  unsigned char* h_out_lp;
  float* y_saved;
  int act, residual;
  int nsl;                     // > 0: aggregate form, sums are the nsl slices below
  const float* slices;         // [nsl][n_dst][d]
};

// y_i = mean_i + Wr h_i + br;  out_i = [h_i +] act(y_i)
template <typename T, int DL>
__global__ __launch_bounds__(256) void k_fwd_node(NodeArgs a) {
  constexpr int NPB = 256 / DL;
  __shared__ float wr[DL][DL + 1];
  __shared__ float hs[NPB][DL];
  stage_square<DL>(wr, a.wr);
  const int li = threadIdx.x / DL, q = threadIdx.x % DL;
  const T* hin = reinterpret_cast<const T*>(a.h_in);
  for (int64_t base = (int64_t)blockIdx.x * NPB; base < a.n_dst; base += (int64_t)gridDim.x * NPB) {
    const int64_t i = base + li;
    const bool ok = i < a.n_dst;
    // every global read of the node is issued ahead of the barriers
    float hv = 0.0f, sum = 0.0f;
    int32_t deg = 0;
    if (ok) {
      hv = to_f(hin[i * DL + q]);
      deg = a.row_ptr[i + 1] - a.row_ptr[i];
      sum = a.nsl > 0 ? ordered_sum(a.slices + i * DL + q, a.n_dst * DL, a.nsl)
                      : segment_sum(a.row_ptr, i, q, DL, a.direct, a.part);
    }
    __syncthreads();
    hs[li][q] = hv;
    __syncthreads();
    if (!ok) continue;
    float y = deg > 0 ? sum / (float)deg : 0.0f;
    float r = 0.0f;
#pragma unroll 8
    for (int p = 0; p < DL; ++p) r += wr[q][p] * hs[li][p];
    y += r + a.br[q];
    const float act = a.act == DSMP_ACT_RELU ? (y > 0.0f ? y : 0.0f) : y;
    const float out = a.residual ? hv + act : act;
    a.h_out[i * DL + q] = out;
    if (a.h_out_lp) reinterpret_cast<T*>(a.h_out_lp)[i * DL + q] = (T)out;
    a.y_saved[i * DL + q] = y;
  }
}

// bf16 layers, d = 64 or 128: the root term on matrix cores,
// C[i][q] = sum_p h_i[p] Wr[q][p] (Wr and h are bf16 values, so the products
// are exact and accumulate in fp32).  A step covers NR = 128 / (d / 32)
// destinations; wave w takes the 32 x 32 block (row tile w / QT, column tile
// w % QT) in the accumulator layout (lane = column q, register r = row
// 8(r/4) + 4h + r%4), so that the sums, h, and the three outputs move as
// whole cache lines across the lanes.  The wave's Wr rows stay in registers.
template <int DL>
__global__ __launch_bounds__(256) void k_fwd_node_m(NodeArgs a) {
  using M = MT<__bf16>;
  constexpr int QT = DL / 32, RT = 4 / QT, NR = 32 * RT, SK = DL / 16;
  const int tid = threadIdx.x, lane = tid & 63, hh = lane >> 5, l32 = lane & 31;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: row bases in scalar registers
  const int rt = wv / QT, ct = wv % QT, q = 32 * ct + l32;
  bf16x8 bw[SK];   // B operand: lane (q, h) holds Wr[q][16s + 8h + t]
#pragma unroll
  for (int s = 0; s < SK; ++s) {
    const float* w = a.wr + (size_t)q * DL + 16 * s + 8 * hh;
    const float4 lo = *reinterpret_cast<const float4*>(w), hi = *reinterpret_cast<const float4*>(w + 4);
    const float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    bw[s] = pack_frag<__bf16>(v);   // exact: the values are bf16 already
  }
  const float brq = a.br[q];
  const __bf16* hin = reinterpret_cast<const __bf16*>(a.h_in);
  const uint32_t lo4 = (uint32_t)(4 * hh * DL + q) * 4u, lo2 = lo4 / 2;
  auto row_of = [&](int r) { return 8 * (r / 4) + 4 * hh + r % 4; };
  // element (row0 + row_of(r), q): a scalar base per row group, the lane offset, a constant per register
  auto at4 = [&](const float* base, int64_t row0, int r) {
    return reinterpret_cast<const float*>(reinterpret_cast<const char*>(base + (row0 + 8 * (r / 4)) * DL) + lo4) +
           (r % 4) * DL;
  };
  auto at2 = [&](const __bf16* base, int64_t row0, int r) {
    return reinterpret_cast<const __bf16*>(reinterpret_cast<const char*>(base + (row0 + 8 * (r / 4)) * DL) + lo2) +
           (r % 4) * DL;
  };
  const int64_t n = a.n_dst;
  for (int64_t b = (int64_t)blockIdx.x * NR; b < n; b += (int64_t)gridDim.x * NR) {
    const int64_t rb = b + 32 * rt;   // first row of the wave's block
    if (rb >= n) continue;            // (wave-uniform) a step past the end
    const bool full = rb + 32 <= n;
    const int rlast = full ? 31 : (int)(n - 1 - rb);
    int degl;   // lane l32: degree of row rb + l32
    {
      const int64_t i = rb + l32 < n ? rb + l32 : n - 1;
      const int32_t d0 = a.row_ptr[i], d1 = a.row_ptr[i + 1];
      degl = d1 - d0;
    }
    bf16x8 A[SK];   // A operand: lane (i, h) holds h_i[16s + 8h + t]
    {
      const int64_t i = rb + (l32 < rlast ? l32 : rlast);
#pragma unroll
      for (int s = 0; s < SK; ++s) A[s] = *reinterpret_cast<const bf16x8*>(hin + i * DL + 16 * s + 8 * hh);
    }
    // h and the sums (the K slices in order, each slice's 16 loads issued together)
    float sum[16], hv[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) sum[r] = 0.0f;
    if (full) {
#pragma unroll
      for (int r = 0; r < 16; ++r) hv[r] = (float)*at2(hin, rb, r);
      for (int k = 0; k < a.nsl; ++k) {
        const float* sk = a.slices + (size_t)k * n * DL;
        float v[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = *at4(sk, rb, r);
#pragma unroll
        for (int r = 0; r < 16; ++r) sum[r] += v[r];
      }
    } else {   // rows past the end re-read the last row
      auto oi = [&](int r) { return (rb + (row_of(r) < rlast ? row_of(r) : rlast)) * DL + q; };
#pragma unroll
      for (int r = 0; r < 16; ++r) hv[r] = (float)hin[oi(r)];
      for (int k = 0; k < a.nsl; ++k) {
        const float* sk = a.slices + (size_t)k * n * DL;
        float v[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = sk[oi(r)];
#pragma unroll
        for (int r = 0; r < 16; ++r) sum[r] += v[r];
      }
    }
    if (a.nsl == 0) {   // per-edge form: tile partial sums
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t i = rb + (row_of(r) < rlast ? row_of(r) : rlast);
        sum[r] = segment_sum(a.row_ptr, i, q, DL, a.direct, a.part);
      }
    }
    f32x16 C = f32x16{};
#pragma unroll
    for (int s = 0; s < SK; ++s) C = M::mma(A[s], bw[s], C);
    const bool relu = a.act == DSMP_ACT_RELU;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      if (!full && row_of(r) > rlast) continue;
      const int deg = __shfl(degl, row_of(r), 64);
      const float y = (deg > 0 ? sum[r] / (float)deg : 0.0f) + (C[r] + brq);
      const float act = relu ? (y > 0.0f ? y : 0.0f) : y;
      const float out = a.residual ? hv[r] + act : act;
      *const_cast<float*>(at4(a.h_out, rb, r)) = out;
      *const_cast<float*>(at4(a.y_saved, rb, r)) = y;
      if (a.h_out_lp) *const_cast<__bf16*>(at2(reinterpret_cast<const __bf16*>(a.h_out_lp), rb, r)) = (__bf16)out;
    }
  }
}

// ------------------------------------------------------------------ kernel MLP

// Layers 1 and 2 of the kernel network K_phi (eq. (1)) for every edge, the
// pass the aggregate form runs ahead of its per-destination sums (bf16
// layers):  z1 = ReLU(W1 x + b1),  z = ReLU(W2 z1 + b2),  with the ReLU mask
// bits of both, and z1 and the split attributes when the backward reads them
// back.  Both layers are matrix-core products over a 32-edge tile:
//  * layer 1 in fp32, 32x32x2 steps over the attribute slots that can be
//    nonzero (two per step), with the bias as the accumulator's initial
//    value: any fp32 evaluation order of the pre-activation is within the
//    accumulation bound the ReLU decisions are held to;
//  * layer 2 in bf16, the bias again the accumulator's initial value.
// W1, W2 (packed columns) and the biases sit in LDS for the workgroup's
// lifetime.
// The layer-1 accumulator rows are the neurons in natural order, which is
// the order the packed-column permutation assigns to the layer-2 B operand:
// each half of a 32-row tile's accumulators is one B fragment as it stands,
// and the mask bits come out in the stored format.  Workgroups are
// persistent; each wave takes every (grid * waves)-th tile.
template <int H>
struct MlpShape {
  static constexpr int WAVES = H <= 128 ? 4 : 8;    // waves per workgroup
  static constexpr int PER_CU = H <= 128 ? 4 : 1;   // workgroups per CU (LDS and registers)
  static constexpr int RT = H / 32, SK = H / 16;    // 32-row output tiles; bf16 K steps
  static constexpr int W2B = H * 2 + 16;            // LDS pitch of a W2 row
  static constexpr int LDS = H * W2B + 10 * H * 4;  // W2; W1 and b1 (packed halves); b2
  static constexpr int MW = H / 64;                 // mask words per lane half and layer
};

template <int H, bool SPLIT>
__global__ __launch_bounds__(64 * MlpShape<H>::WAVES, MlpShape<H>::PER_CU) void k_edge_mlp(EdgeArgs a,
                                                                                         int64_t ntiles) {
  using S = MlpShape<H>;
  using M = MT<__bf16>;
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* w2s = smem;
  float* w1s = reinterpret_cast<float*>(smem + H * S::W2B);
  float* b1s = w1s + 8 * H;
  float* b2s = b1s + H;
  const int tid = threadIdx.x, lane = tid & 63, hh = lane >> 5, l32 = lane & 31;
  const unsigned char* P = a.packed;

  // W2, W1 and the biases to LDS, once per workgroup
  {
    constexpr int NU = H * 2 / 16;
    const uint4* src = reinterpret_cast<const uint4*>(P + a.L.w2p);
    for (int U = tid; U < H * NU; U += 64 * S::WAVES)
      *reinterpret_cast<uint4*>(w2s + (U / NU) * S::W2B + (U % NU) * 16) = src[U];
    const uint4* w1l = reinterpret_cast<const uint4*>(P + a.L.w1l);
    for (int U = tid; U < 2 * H; U += 64 * S::WAVES) reinterpret_cast<uint4*>(w1s)[U] = w1l[U];
    const float* b1l = reinterpret_cast<const float*>(P + a.L.b1l);
    const float* b2 = reinterpret_cast<const float*>(P + a.L.b2);
    for (int U = tid; U < H; U += 64 * S::WAVES) {
      b1s[U] = b1l[U];
      b2s[U] = b2[U];
    }
  }
  // Layer-1 A operand: W1[32 rt + l32][2 ks + hh] from the packed halves
  // (neuron 32c + r sits in half (r/4)%2 at position 16c + 4(r/8) + r%4).
  const int nks = attr_slots(a.dim, a.attr_mode) / 2;
  const float* w1a = w1s + ((((l32 >> 2) & 1) * (H / 2) + 4 * (l32 >> 3) + (l32 & 3)) * 8 + hh);
  __syncthreads();

  const int64_t stride = (int64_t)gridDim.x * S::WAVES;
  int64_t tile = (int64_t)blockIdx.x * S::WAVES + (tid >> 6);
  if (tile >= ntiles) return;
  // Loads run a tile ahead: a tile's attribute rows, and the ids of the tile
  // after it, are issued before the stores of the tile in hand, so waiting
  // for them never waits for those stores (loads and stores retire in one
  // in-order count).  Lanes past E read edge 0 and store into the padding
  // rows of the last tile.
  const int rw = a.dim + 1;
  const float* na = a.node_attr;
  auto eid = [&](int64_t t) -> int64_t {
    const int64_t e = t * 32 + l32;
    return e < a.E ? e : 0;
  };
  float ri[4], rj[4];
  auto load_rows = [&](int i, int j) {
    const float* pi = na + (size_t)i * rw;
    const float* pj = na + (size_t)j * rw;
    ri[0] = pi[0]; ri[1] = pi[1]; ri[2] = pi[2];
    rj[0] = pj[0]; rj[1] = pj[1]; rj[2] = pj[2];
    ri[3] = rw == 4 ? pi[3] : 0.0f;
    rj[3] = rw == 4 ? pj[3] : 0.0f;
  };
  {
    const int64_t e0 = eid(tile);
    load_rows(a.dst[e0], a.col[e0]);
  }
  int ni, nj;
  {
    const int64_t e1 = eid(tile + stride);
    ni = a.dst[e1];
    nj = a.col[e1];
  }

  // The loop is re-entered with a tile's stores issued after the next tile's
  // loads.  The compiler's wait counts at the loop head take the smaller count
  // of its two ways in, so the way in from here issues as many stores after
  // those loads, into the spare mask rows past the last tile (never read).
  {
    constexpr int NST = 2 * S::RT + 2 + (SPLIT ? S::SK + 1 : 0);
    constexpr int RW = 2 * H / 32;   // mask words per edge
    uint32_t* sink = reinterpret_cast<uint32_t*>(a.zmask + (size_t)ntiles * 32 * RW * 4);
    // a lane-dependent row per store keeps them from merging into wider ones
#pragma unroll
    for (int k = 0; k < NST; ++k) sink[((l32 + 5 * k) % 32) * RW + (k / 32) % RW] = 0u;
  }
  for (; tile < ntiles; tile += stride) {
    const int64_t e = tile * 32 + l32;
    float x[8];
    edge_attr_rows(ri, rj, a.dim, a.attr_mode, x);
    load_rows(ni, nj);
    {
      const int64_t e2 = eid(tile + 2 * stride);
      ni = a.dst[e2];
      nj = a.col[e2];
    }
    if constexpr (SPLIT) {   // bf16 high parts (lane half 0), then low parts (half 1)
      float v[8];
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const float hi = (float)(__bf16)x[c];
        v[c] = hh ? x[c] - hi : hi;
      }
      *reinterpret_cast<bf16x8*>(a.xE + (size_t)e * 32 + hh * 16) = pack_frag<__bf16>(v);
    }
    // B operand of layer 1: slot 2 ks + hh of the lane's edge (the values go
    // through registers first, so the choice stays a select of values)
    float xb[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      float x0 = x[2 * ks], x1 = x[2 * ks + 1];
      asm("" : "+v"(x0), "+v"(x1));
      xb[ks] = hh ? x1 : x0;
    }

    // layer 1
    bf16x8 z1B[S::SK];
    uint32_t m1[S::MW], m2[S::MW];
#pragma unroll
    for (int w = 0; w < S::MW; ++w) m1[w] = m2[w] = 0u;
#pragma unroll
    for (int rt = 0; rt < S::RT; ++rt) {
      f32x16 C;
      const f32x4* bp = reinterpret_cast<const f32x4*>(b1s + hh * (H / 2) + 16 * rt);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x4 b = bp[q];
        C[4 * q] = b[0]; C[4 * q + 1] = b[1]; C[4 * q + 2] = b[2]; C[4 * q + 3] = b[3];
      }
      const float* w1t = w1a + 16 * rt * 8;
      C = MT<float>::mma(w1t[0], xb[0], C);
      C = MT<float>::mma(w1t[2], xb[1], C);
      if (nks > 2) C = MT<float>::mma(w1t[4], xb[2], C);
      if (nks > 3) C = MT<float>::mma(w1t[6], xb[3], C);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        float zv[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int b = (2 * rt + j) * 8 + t;
          zv[t] = relu_mask(C[8 * j + t], m1[b / 32], b % 32);
        }
        z1B[2 * rt + j] = pack_frag<__bf16>(zv);
      }
      // fold the tile's mask bits into their words here rather than at the store
#pragma unroll
      for (int w = 0; w < S::MW; ++w) asm("" : "+v"(m1[w]));
    }
    if constexpr (SPLIT) {
      if (a.z1E) {   // without z1 rows the backward recomputes z1 from the split attributes
#pragma unroll
        for (int s = 0; s < S::SK; ++s)
          *reinterpret_cast<bf16x8*>(a.z1E + ((size_t)e * H + s * 16 + hh * 8) * 2) = z1B[s];
      }
    }

    // layer 2, one 32-row tile of outputs at a time
#pragma unroll
    for (int kt = 0; kt < S::RT; ++kt) {
      f32x16 C;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x4 b = *reinterpret_cast<const f32x4*>(b2s + kt * 32 + 8 * q + 4 * hh);
        C[4 * q] = b[0]; C[4 * q + 1] = b[1]; C[4 * q + 2] = b[2]; C[4 * q + 3] = b[3];
      }
#pragma unroll
      for (int s = 0; s < S::SK; ++s) {
        const bf16x8 A = *reinterpret_cast<const bf16x8*>(w2s + (kt * 32 + l32) * S::W2B + (s * 16 + hh * 8) * 2);
        C = M::mma(A, z1B[s], C);
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        float zv[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int b = 16 * kt + 8 * j + t;
          zv[t] = relu_mask(C[8 * j + t], m2[b / 32], b % 32);
        }
        *reinterpret_cast<bf16x8*>(a.zE + ((size_t)e * H + (2 * kt + j) * 16 + hh * 8) * 2) =
            pack_frag<__bf16>(zv);
      }
#pragma unroll
      for (int w = 0; w < S::MW; ++w) asm("" : "+v"(m2[w]));
    }
    uint32_t* mb = reinterpret_cast<uint32_t*>(a.zmask + (size_t)e * (2 * H / 8));
#pragma unroll
    for (int w = 0; w < S::MW; ++w) mb[hh * S::MW + w] = m1[w];
#pragma unroll
    for (int w = 0; w < S::MW; ++w) mb[2 * S::MW + hh * S::MW + w] = m2[w];
  }
}

template <int H>
dsmp_status launch_edge_mlp(dsmp_handle* h, const EdgeArgs& a) {
  using S = MlpShape<H>;
  DSMP_CHECK(h, a.zE != nullptr && a.zmask != nullptr && (a.z1E == nullptr || a.xE != nullptr),
             DSMP_INVALID_ARG, "kernel MLP: z and the mask bits are always stored, z1 only with x");
  auto kern = a.xE ? k_edge_mlp<H, true> : k_edge_mlp<H, false>;
  DSMP_HIP(h, hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, S::LDS));
  const int64_t ntiles = ceil_div(a.E, 32);
  const int64_t grid = std::min<int64_t>(ceil_div(ntiles, S::WAVES), (int64_t)h->n_cu * S::PER_CU);
  ProfScope prof(h, DSMP_K_EDGE_MLP);
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(64 * S::WAVES), S::LDS, h->stream, a, ntiles);
  DSMP_LAUNCHED(h, "kernel MLP");
  return DSMP_OK;
}


// ------------------------------------------------------------------ packing

struct PackArgs {
  const float *W1, *b1, *W2, *b2, *W3, *b3, *Wr, *br;
  int d, h1, h2, de;
  PackLayout L;
  unsigned char* out;
  int nloop;   // workgroups of the element loops; d * ceil(h2/32) more transpose W3 tiles
};

// The two packed forms of W3 [p][q][k] that put q fastest, through an LDS
// tile so that both the reads (rows of k) and the writes (rows of q) are
// whole cache lines; one workgroup per tile (32 values of k, p), tb:
//  * w3t [p][k][q];
//  * W3u, the U GEMM's B operand, rows in MFMA fragment order: row c of W3u
//    is U_i's element (k, p) that lane l of A fragment (kt, s) holds,
//    c = ((kt*SKD + s)*64 + l)*EPL + t, with k = 32 kt + l%32 and
//    p = s*KS + (l/32)*EPL + t, so a fragment of U_i is one contiguous
//    64-lane piece.
template <typename T>
__device__ __forceinline__ void pack_w3_tile(const float* __restrict__ W3, int d, int h2, int tb,
                                             T* __restrict__ w3t, T* __restrict__ w3u) {
  constexpr int KS = MT<T>::KS, EPL = MT<T>::EPL, MAXU = 128 * 32 / 256;   // d <= 128
  __shared__ float tile[32][129];   // [k - k0][q]
  const int nkb = (h2 + 31) / 32, tid = threadIdx.x;
  const int k0 = (tb % nkb) * 32, p = tb / nkb;
  float v[MAXU];   // every load of the tile issued before the first LDS write
#pragma unroll
  for (int i = 0; i < MAXU; ++i) {
    const int u = tid + 256 * i, q = u / 32, kk = u % 32;
    v[i] = u < d * 32 && k0 + kk < h2 ? W3[((int64_t)p * d + q) * h2 + k0 + kk] : 0.0f;
  }
#pragma unroll
  for (int i = 0; i < MAXU; ++i) {
    const int u = tid + 256 * i;
    if (u < d * 32) tile[u % 32][u / 32] = v[i];
  }
  __syncthreads();
  const int skd = d / KS, t = p % EPL, s = p / KS, lh = (p % KS) / EPL;
  for (int u = tid; u < d * 32; u += 256) {
    const int kk = u / d, q = u % d, k = k0 + kk;
    if (k >= h2) continue;
    const T x = (T)tile[kk][q];
    w3t[((int64_t)p * h2 + k) * d + q] = x;
    const int l = lh * 32 + k % 32, fs = (k / 32) * skd + s;
    w3u[((int64_t)(fs * 64 + l) * EPL + t) * d + q] = x;
  }
}

template <typename T>
__global__ void k_pack(PackArgs a) {
  constexpr int KS = MT<T>::KS, EPL = MT<T>::EPL;
  const int d = a.d, h1 = a.h1, h2 = a.h2;
  if ((int)blockIdx.x >= a.nloop) {   // the blocks past the element loops' grid transpose one W3 tile each
    pack_w3_tile<T>(a.W3, d, h2, (int)blockIdx.x - a.nloop, reinterpret_cast<T*>(a.out + a.L.w3t),
                    reinterpret_cast<T*>(a.out + a.L.w3u));
    return;
  }
  const int64_t stride = (int64_t)a.nloop * blockDim.x;
  const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  float* w1l = reinterpret_cast<float*>(a.out + a.L.w1l);
  float* b1l = reinterpret_cast<float*>(a.out + a.L.b1l);
  for (int64_t x = t0; x < (int64_t)h1 * 8; x += stride) {
    int c = x % 8, hn = x / 8, hh = hn / (h1 / 2), n = hn % (h1 / 2);
    int j = kperm<T>((n / EPL) * KS + hh * EPL + n % EPL);
    w1l[x] = c < a.de ? a.W1[j * a.de + c] : 0.0f;
    if (c == 0) b1l[hn] = a.b1[j];
  }
  T* w2p = reinterpret_cast<T*>(a.out + a.L.w2p);
  T* w2t = reinterpret_cast<T*>(a.out + a.L.w2t);
  for (int64_t x = t0; x < (int64_t)h2 * h1; x += stride) {
    int k = x / h1, kk = x % h1;
    w2p[x] = (T)a.W2[k * h1 + kperm<T>(kk)];
    int j = x / h2, kk2 = x % h2;
    w2t[x] = (T)a.W2[kperm<T>(kk2) * h1 + j];
  }
  float* b2 = reinterpret_cast<float*>(a.out + a.L.b2);
  for (int64_t x = t0; x < h2; x += stride) b2[x] = a.b2[x];
  T* w3f = reinterpret_cast<T*>(a.out + a.L.w3f);
  T* w3q = reinterpret_cast<T*>(a.out + a.L.w3q);
  for (int64_t x = t0; x < (int64_t)d * d * h2; x += stride) {
    int64_t r = x / h2;
    int kk = x % h2;
    int i0 = r / d, i1 = r % d;
    // w3f[p=i0][q=i1][kk], w3q[q=i0][p=i1][kk]
    w3f[x] = (T)a.W3[((int64_t)i0 * d + i1) * h2 + kperm<T>(kk)];
    w3q[x] = (T)a.W3[((int64_t)i1 * d + i0) * h2 + kperm<T>(kk)];
  }
  T* b3t = reinterpret_cast<T*>(a.out + a.L.b3t);
  T* b3n = reinterpret_cast<T*>(a.out + a.L.b3n);
  float* wr = reinterpret_cast<float*>(a.out + a.L.wr);
  for (int64_t x = t0; x < (int64_t)d * d; x += stride) {
    int i0 = x / d, i1 = x % d;
    b3t[x] = (T)a.b3[i1 * d + i0];
    b3n[x] = (T)a.b3[x];
    wr[x] = (float)(T)a.Wr[x];
  }
  float* br = reinterpret_cast<float*>(a.out + a.L.br);
  for (int64_t x = t0; x < d; x += stride) br[x] = a.br[x];
  // W3~ in the segment-sum K order: K < h2*d is (k stored position, c) of a
  // 32x32 accumulator tile, K = h2*d + c is the bias row.
  T* wgt = reinterpret_cast<T*>(a.out + a.L.wgt);
  T* wht = reinterpret_cast<T*>(a.out + a.L.wht);
  const int64_t ktot = (int64_t)h2 * d + d;
  const int nct = d / 32;
  for (int64_t x = t0; x < (int64_t)d * ktot; x += stride) {
    const int o = (int)(x / ktot);
    const int64_t K = x % ktot;
    if (K < (int64_t)h2 * d) {
      const int ti = (int)(K / 1024), rem = (int)(K % 1024), l = rem / 16, r = rem % 16;
      const int kpos = (ti / nct) * 32 + 8 * (r / 4) + 4 * (l / 32) + (r % 4);
      const int c = (ti % nct) * 32 + (l % 32);
      const int k = kperm<T>(kpos);
      wgt[x] = (T)a.W3[((int64_t)c * d + o) * h2 + k];   // output q = o, sum column p = c
      wht[x] = (T)a.W3[((int64_t)o * d + c) * h2 + k];   // output p = o, sum column q = c
    } else {
      const int c = (int)(K - (int64_t)h2 * d);
      wgt[x] = (T)a.b3[c * d + o];
      wht[x] = (T)a.b3[o * d + c];
    }
  }
}

template <typename K>
dsmp_status set_lds(dsmp_handle* h, K kernel, int bytes) {
  DSMP_HIP(h, hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, bytes));
  return DSMP_OK;
}

template <typename T, int DL, int H1, int H2>
dsmp_status launch_edge_shape(dsmp_handle* h, int mode, const EdgeArgs& a) {
  using S = Shape<T, DL, H1, H2>;
  const unsigned grid = ceil_div(a.E, S::TILE);
  if (mode == MODE_FWD) {
    auto kern = k_edge_contract<T, DL, H1, H2, MODE_FWD>;
    dsmp_status st = set_lds(h, kern, S::LDS);
    if (st != DSMP_OK) return st;
    ProfScope prof(h, DSMP_K_EDGE_FWD);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(256), S::LDS, h->stream, a);
  } else if (mode == MODE_MLP) {
    if constexpr (sizeof(T) == 2 && H1 == H2) {
      return launch_edge_mlp<H1>(h, a);
    } else {
      auto kern = k_edge_contract<T, DL, H1, H2, MODE_MLP>;
      dsmp_status st = set_lds(h, kern, S::LDS);
      if (st != DSMP_OK) return st;
      ProfScope prof(h, DSMP_K_EDGE_MLP);
      hipLaunchKernelGGL(kern, dim3(grid), dim3(256), S::LDS, h->stream, a);
    }
  } else {
    auto kern = k_edge_contract<T, DL, H1, H2, MODE_DH>;
    dsmp_status st = set_lds(h, kern, S::LDS);
    if (st != DSMP_OK) return st;
    ProfScope prof(h, DSMP_K_EDGE_DH);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(256), S::LDS, h->stream, a);
  }
  DSMP_LAUNCHED(h, "edge contraction");
  return DSMP_OK;
}

}  // namespace

namespace dsmp {

bool shape_supported(const dsmp_layer_desc& d) {
  if (d.dtype == DSMP_F32) return (d.d == 32 && d.h1 == 64 && d.h2 == 64) ||
                                  (d.d == 64 && d.h1 == 128 && d.h2 == 128);
  if (d.dtype == DSMP_BF16) return (d.d == 32 && d.h1 == 64 && d.h2 == 64) ||
                                   (d.d == 64 && d.h1 == 128 && d.h2 == 128) ||
                                   (d.d == 128 && d.h1 == 256 && d.h2 == 256);
  return false;
}

dsmp_status launch_edge_contract(dsmp_handle* h, const dsmp_layer_desc& d, int mode,
                                 const EdgeArgs& a) {
  if (a.E == 0) return DSMP_OK;
  if (d.dtype == DSMP_F32) {
    if (d.d == 32) return launch_edge_shape<float, 32, 64, 64>(h, mode, a);
    if (d.d == 64) return launch_edge_shape<float, 64, 128, 128>(h, mode, a);
  } else {
    if (d.d == 32) return launch_edge_shape<__bf16, 32, 64, 64>(h, mode, a);
    if (d.d == 64) return launch_edge_shape<__bf16, 64, 128, 128>(h, mode, a);
    if (d.d == 128) return launch_edge_shape<__bf16, 128, 256, 256>(h, mode, a);
  }
  return fail(h, DSMP_UNSUPPORTED, "unsupported layer shape");
}

}  // namespace dsmp

// ------------------------------------------------------------------ C ABI

namespace {

int attr_width(const dsmp_layer_desc& d) {
  return d.attr_mode == DSMP_ATTR_CONCAT ? 2 * d.dim + 2 : d.dim + 1;
}

dsmp_status check_desc(dsmp_handle* h, const dsmp_layer_desc* d) {
  DSMP_CHECK(h, d != nullptr, DSMP_INVALID_ARG, "layer descriptor is NULL");
  DSMP_CHECK(h, d->dim == 2 || d->dim == 3, DSMP_INVALID_ARG, "dim must be 2 or 3");
  DSMP_CHECK(h, d->dtype == DSMP_F32 || d->dtype == DSMP_BF16, DSMP_INVALID_ARG, "unknown dtype");
  DSMP_CHECK(h, d->act == DSMP_ACT_IDENTITY || d->act == DSMP_ACT_RELU, DSMP_INVALID_ARG,
             "unknown activation");
  DSMP_CHECK(h, d->attr_mode == DSMP_ATTR_CONCAT || d->attr_mode == DSMP_ATTR_DIFF, DSMP_INVALID_ARG,
             "unknown edge attribute mode");
  DSMP_CHECK(h, d->residual == 0 || d->residual == 1, DSMP_INVALID_ARG, "residual must be 0 or 1");
  DSMP_CHECK(h, shape_supported(*d), DSMP_UNSUPPORTED,
             "unsupported widths d=%d h1=%d h2=%d for this dtype", d->d, d->h1, d->h2);
  return DSMP_OK;
}

}  // namespace

namespace dsmp {

dsmp_status check_layer_desc(dsmp_handle* h, const dsmp_layer_desc* d) { return check_desc(h, d); }
int layer_attr_width(const dsmp_layer_desc& d) { return attr_width(d); }

SavedLayout saved_layout(const dsmp_layer_desc& d, int64_t n_dst, int64_t E) {
  Carve c(nullptr);
  int esz = d.dtype == DSMP_BF16 ? 2 : 4;
  SavedLayout s;
  s.y = (size_t)c.take<float>((size_t)n_dst * d.d) ;
  // per-edge sections hold whole 32-edge tiles: the kernel-MLP pass stores
  // its last tile's rows past E without a per-lane condition; the mask bits
  // have one more tile of rows that it writes and nothing reads
  const int64_t E32 = (E + 31) / 32 * 32;
  s.zE = (size_t)c.take<unsigned char>((size_t)E32 * d.h2 * esz);
  s.z1E = (size_t)c.take<unsigned char>((size_t)E32 * d.h1 * esz);
  s.zmask = (size_t)c.take<unsigned char>((size_t)(E32 + 32) * (d.h1 + d.h2) / 8);
  s.xE = (size_t)c.take<unsigned char>(d.dtype == DSMP_BF16 ? (size_t)E32 * 32 : 0);
  s.os = (size_t)c.take<unsigned char>((size_t)n_dst * agg_ktot(d) * esz + 512);   // + whole last staged piece
  s.total = c.used();
  return s;
}

size_t fwd_ws_bytes(const dsmp_layer_desc& d, int64_t n_dst, int64_t E) {
  // per-edge form: direct sums and tile partials; aggregate form: GEMM slices
  Carve c(nullptr);
  c.take<float>((size_t)n_dst * d.d);
  c.take<float>((size_t)(ceil_div(E, EDGE_TILE) + 1) * 2 * d.d);
  const size_t per_edge = c.used();
  Carve c2(nullptr);
  c2.take<float>((size_t)agg_gemm_slices(n_dst, d) * n_dst * d.d);
  return per_edge > c2.used() ? per_edge : c2.used();
}

dsmp_status check_graph(dsmp_handle* h, const dsmp_graph* g, bool need_csc) {
  DSMP_CHECK(h, g != nullptr, DSMP_INVALID_ARG, "graph is NULL");
  DSMP_CHECK(h, g->n_dst >= 0 && g->n_src >= g->n_dst && g->n_edges >= 0, DSMP_INVALID_ARG,
             "bad graph sizes");
  DSMP_CHECK(h, g->n_edges <= INT32_MAX && g->n_src <= INT32_MAX, DSMP_UNSUPPORTED,
             "graph too large for int32 indices");
  DSMP_CHECK(h, g->row_ptr != nullptr, DSMP_INVALID_ARG, "row_ptr is NULL");
  DSMP_CHECK(h, g->n_edges == 0 || (g->col && g->dst), DSMP_INVALID_ARG, "col or dst is NULL");
  if (need_csc)
    DSMP_CHECK(h, g->csc_ptr && (g->n_edges == 0 || g->csc_eid), DSMP_INVALID_ARG,
               "csc arrays are NULL");
  return DSMP_OK;
}

}  // namespace dsmp

extern "C" dsmp_status dsmp_nnconv_packed_bytes(const dsmp_layer_desc* desc, size_t* bytes) {
  if (!desc || !bytes) return DSMP_INVALID_ARG;
  dsmp_status st = check_desc(nullptr, desc);
  if (st != DSMP_OK) return st;
  *bytes = pack_layout(desc->d, desc->h1, desc->h2, desc->dtype == DSMP_BF16 ? 2 : 4).total;
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_nnconv_pack(dsmp_handle* h, const dsmp_layer_desc* desc,
                                        const dsmp_layer_params* p, void* packed) {
  if (!h) return DSMP_INVALID_ARG;
  dsmp_status st = check_desc(h, desc);
  if (st != DSMP_OK) return st;
  DSMP_CHECK(h, p && p->W1 && p->b1 && p->W2 && p->b2 && p->W3 && p->b3 && p->Wr && p->br && packed,
             DSMP_INVALID_ARG, "a parameter pointer is NULL");
  DSMP_CHECK(h, (reinterpret_cast<uintptr_t>(packed) & 255) == 0, DSMP_INVALID_ARG,
             "packed buffer must be 256-byte aligned");
  PackArgs a{p->W1, p->b1, p->W2, p->b2, p->W3, p->b3, p->Wr, p->br,
             desc->d, desc->h1, desc->h2, attr_width(*desc),
             pack_layout(desc->d, desc->h1, desc->h2, desc->dtype == DSMP_BF16 ? 2 : 4),
             static_cast<unsigned char*>(packed), 1024};
  const dim3 grid((unsigned)(a.nloop + desc->d * ceil_div(desc->h2, 32)));
  if (desc->dtype == DSMP_BF16)
    hipLaunchKernelGGL(k_pack<__bf16>, grid, dim3(256), 0, h->stream, a);
  else
    hipLaunchKernelGGL(k_pack<float>, grid, dim3(256), 0, h->stream, a);
  DSMP_LAUNCHED(h, "pack");
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_nnconv_forward(dsmp_handle* h, const dsmp_layer_desc* desc,
                                           const void* packed, const dsmp_graph* g,
                                           const float* node_attr, const void* h_in, float* h_out,
                                           void* h_out_lp, void* saved, size_t saved_bytes, void* ws,
                                           size_t ws_bytes) {
  if (!h) return DSMP_INVALID_ARG;
  dsmp_status st = check_desc(h, desc);
  if (st != DSMP_OK) return st;
  if ((st = check_graph(h, g, false)) != DSMP_OK) return st;
  const dsmp_layer_desc& d = *desc;
  DSMP_CHECK(h, packed && (g->n_src == 0 || (node_attr && h_in)) && (g->n_dst == 0 || h_out),
             DSMP_INVALID_ARG, "a forward pointer is NULL");
  SavedLayout sl = saved_layout(d, g->n_dst, g->n_edges);
  size_t need_ws = fwd_ws_bytes(d, g->n_dst, g->n_edges);
  DSMP_CHECK(h, saved && saved_bytes >= sl.total, DSMP_WORKSPACE_TOO_SMALL,
             "saved buffer needs %zu bytes", sl.total);
  DSMP_CHECK(h, ws && ws_bytes >= need_ws, DSMP_WORKSPACE_TOO_SMALL, "forward workspace needs %zu bytes",
             need_ws);
  const int esz = d.dtype == DSMP_BF16 ? 2 : 4;
  PackLayout L = pack_layout(d.d, d.h1, d.h2, esz);
  unsigned char* sv = static_cast<unsigned char*>(saved);
  const bool agg = use_aggregate(h, d, g->n_dst, g->n_edges);
  Carve c(ws);
  float *direct = nullptr, *part = nullptr, *slices = nullptr;
  int nsl = 0;
  if (agg) {
    nsl = agg_gemm_slices(g->n_dst, d);
    slices = c.take<float>((size_t)nsl * g->n_dst * d.d);
  } else {
    direct = c.take<float>((size_t)g->n_dst * d.d);
    part = c.take<float>((size_t)(ceil_div(g->n_edges, EDGE_TILE) + 1) * 2 * d.d);
  }
  EdgeArgs ea{};
  ea.E = g->n_edges; ea.n_dst = g->n_dst; ea.n_src = g->n_src;
  ea.row_ptr = g->row_ptr; ea.col = g->col; ea.dst = g->dst;
  ea.node_attr = node_attr; ea.dim = d.dim; ea.attr_mode = d.attr_mode;
  ea.gath = static_cast<const unsigned char*>(h_in);
  ea.packed = static_cast<const unsigned char*>(packed); ea.L = L;
  ea.zE = sv + sl.zE; ea.z1E = sv + sl.z1E; ea.zmask = sv + sl.zmask;
  ea.xE = d.dtype == DSMP_BF16 ? sv + sl.xE : nullptr;
  if (agg && fused_edge_grads(d)) ea.z1E = ea.xE = nullptr;   // the backward recomputes both
  if (dz_with_m(d, agg)) ea.z1E = nullptr;                     // the dW2 pass recomputes z1 from x
  ea.out_direct = direct; ea.out_part = part;
  if (agg) {
    // z and z1 per edge, the per-destination sums S (kept for the backward),
    // then one GEMM with W3~ into nsl K-slices
    if ((st = launch_edge_contract(h, d, MODE_MLP, ea)) != DSMP_OK) return st;
    {
      ProfScope prof(h, DSMP_K_OUTER_FWD);
      st = launch_outer_sum(h, d, g->n_dst, g->row_ptr, nullptr, g->col, sv + sl.zE,
                            static_cast<const unsigned char*>(h_in), sv + sl.os);
    }
    if (st != DSMP_OK) return st;
    {
      ProfScope prof(h, DSMP_K_GEMM_FWD);
      st = launch_w3_gemm(h, d, g->n_dst, sv + sl.os, ea.packed + L.wgt, nsl, slices);
    }
    if (st != DSMP_OK) return st;
  } else {
    if ((st = launch_edge_contract(h, d, MODE_FWD, ea)) != DSMP_OK) return st;
  }
  if (g->n_dst > 0) {
    NodeArgs na{g->n_dst, g->row_ptr, static_cast<const unsigned char*>(h_in), direct, part,
                reinterpret_cast<const float*>(ea.packed + L.wr),
                reinterpret_cast<const float*>(ea.packed + L.br), h_out,
                static_cast<unsigned char*>(h_out_lp), reinterpret_cast<float*>(sv + sl.y), d.act,
                d.residual, nsl, slices};
    unsigned grid = ceil_div(g->n_dst, 256 / d.d);
    if (grid > 2048) grid = 2048;
    ProfScope prof(h, DSMP_K_NODE_FWD);
    if (d.dtype == DSMP_BF16) {
      if (d.d == 32) hipLaunchKernelGGL((k_fwd_node<__bf16, 32>), dim3(grid), dim3(256), 0, h->stream, na);
      // matrix-core root term (steps of 128 / (d / 32) destinations) where
      // there are enough steps to fill the CUs; the LDS form otherwise
      const int64_t nstep = ceil_div(g->n_dst, 128 / (d.d / 32));
      const unsigned gm = (unsigned)std::min<int64_t>(nstep, (int64_t)h->n_cu * 8);
      const bool mfma_root = nstep >= (int64_t)h->n_cu * 2;
      if (d.d == 64 && mfma_root) hipLaunchKernelGGL((k_fwd_node_m<64>), dim3(gm), dim3(256), 0, h->stream, na);
      if (d.d == 64 && !mfma_root) hipLaunchKernelGGL((k_fwd_node<__bf16, 64>), dim3(grid), dim3(256), 0, h->stream, na);
      if (d.d == 128 && mfma_root) hipLaunchKernelGGL((k_fwd_node_m<128>), dim3(gm), dim3(256), 0, h->stream, na);
      if (d.d == 128 && !mfma_root)
        hipLaunchKernelGGL((k_fwd_node<__bf16, 128>), dim3(grid), dim3(256), 0, h->stream, na);
    } else {
      if (d.d == 32) hipLaunchKernelGGL((k_fwd_node<float, 32>), dim3(grid), dim3(256), 0, h->stream, na);
      if (d.d == 64) hipLaunchKernelGGL((k_fwd_node<float, 64>), dim3(grid), dim3(256), 0, h->stream, na);
    }
    DSMP_LAUNCHED(h, "forward node update");
  }
  return DSMP_OK;
}
