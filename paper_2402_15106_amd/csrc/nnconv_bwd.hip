// NNConv layer backward: gradients of the forward in nnconv_fwd.hip with
// respect to the input features and every parameter (the backpropagation step
// of Algorithm 1 for one graph-convolution hop).
//
// With ybar = G * act'(y) and the per-edge message gradient g_e = ybar_i/deg_i
// (i the destination of e):
//   dWr = sum_i ybar_i h_i^T,  dbr = sum_i ybar_i,  dh_i += [G_i] + Wr^T ybar_i
//   dh_j += sum_{e: j->i} Theta_e g_e        (edge contraction in source order)
//   dz_e[k] = sum_p h_j[p] sum_q W3[p*d+q][k] g_e[q]   (MFMA, scaled by h_j[p])
//   dW3[p*d+q][k] = sum_e h_j[p] g_e[q] z_e[k],  db3[p*d+q] = sum_e h_j[p] g_e[q]
//   da2 = dz * [z > 0]:  dW2 = sum_e da2 z1^T, db2 = sum_e da2, dz1 = W2^T da2
//   da1 = dz1 * [z1 > 0]: dW1 = sum_e da1 x_e^T, db1 = sum_e da1
// Every sum over edges or nodes is split into fixed chunks whose partial sums
// are added in chunk order: no atomics, bitwise-reproducible results.
#include "nnconv.hpp"

#include <type_traits>

using namespace dsmp;

namespace {

template <typename T>
__device__ __forceinline__ void set_el(typename MT<T>::frag& f, int i, float v);
template <>
__device__ __forceinline__ void set_el<__bf16>(bf16x8& f, int i, float v) { f[i] = (__bf16)v; }
template <>
__device__ __forceinline__ void set_el<float>(float& f, int, float v) { f = v; }

template <typename T>
__device__ __forceinline__ float get_el(const typename MT<T>::frag& f, int i);
template <>
__device__ __forceinline__ float get_el<__bf16>(const bf16x8& f, int i) { return (float)f[i]; }
template <>
__device__ __forceinline__ float get_el<float>(const float& f, int) { return f; }

template <typename T>
__device__ __forceinline__ typename MT<T>::frag ld_frag(const void* p) {
  return *reinterpret_cast<const typename MT<T>::frag*>(p);
}

// A fragment that is zero where !valid.  The load itself is unconditional (p
// must be readable either way): a load under a condition compiles to a branch
// around it, and past such joins the compiler's wait counts fall back to
// waiting for every outstanding load, the loads issued ahead included.
template <typename T>
__device__ __forceinline__ typename MT<T>::frag ld_frag_if(const void* p, bool valid) {
  const typename MT<T>::frag v = ld_frag<T>(p);
  return valid ? v : typename MT<T>::frag{};
}

__device__ __forceinline__ float to_f(__bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f(float x) { return x; }


// ------------------------------------------------------------ node pre-pass

struct BNodeArgs {
  int64_t n_dst, per_block;    // destinations, and destinations per workgroup
  const int32_t* row_ptr;
  const float* G;
  const float* y;
  const float* wr;       // [q][p]
  const unsigned char* h_in;   // [n_src][d] layer dtype
  unsigned char* gT;     // [n_dst][d] layer dtype
  float* gF;             // [n_dst][d]
  float* dh_node;
  float* p_root;         // [grid][d*d + d] partial sums of dWr and dbr
  int act, residual;
};

// The node terms of the backward for a chunk of per_block destinations per
// workgroup, 32 at a time:  ybar_i = G_i * act'(y_i), the message gradient
// g_i = ybar_i / deg_i (fp32 and layer dtype), dh_node_i = [G_i] + Wr^T ybar_i,
// and the workgroup's partial sums dWr = sum_i ybar_i h_i^T, dbr = sum_i ybar_i
// (added over workgroups in a fixed order later).
template <typename T, int DL>
__global__ __launch_bounds__(256) void k_bwd_node(BNodeArgs a) {
  constexpr int NB = 32, NU = NB * DL / 256, PP = DL * DL / 256, NPW = 256 / DL;
  __shared__ float wr[DL][DL + 1];
  __shared__ float ys[NB][DL];
  __shared__ float hs[NB][DL];
  stage_square<DL>(wr, a.wr);
  const int tid = threadIdx.x, c = tid % DL, li = tid / DL;   // element k: node li + NPW*k, column c
  const int q = tid % DL, p0 = (tid / DL) * PP;               // partial sums dWr[q][p0 .. p0+PP)
  const T* hin = reinterpret_cast<const T*>(a.h_in);
  float acc[PP];
#pragma unroll
  for (int u = 0; u < PP; ++u) acc[u] = 0.0f;
  float accb = 0.0f;
  const int64_t i0 = (int64_t)blockIdx.x * a.per_block;
  const int64_t i1 = i0 + a.per_block < a.n_dst ? i0 + a.per_block : a.n_dst;
  for (int64_t b = i0; b < i1; b += NB) {
    float g[NU], v[NU], hv[NU];
    int32_t deg[NU];
#pragma unroll
    for (int k = 0; k < NU; ++k) {
      const int64_t i = b + li + NPW * k;
      g[k] = 0.0f; v[k] = 0.0f; hv[k] = 0.0f; deg[k] = 0;
      if (i < i1) {
        g[k] = a.G[i * DL + c];
        const float yv = a.y[i * DL + c];
        hv[k] = to_f(hin[i * DL + c]);
        deg[k] = a.row_ptr[i + 1] - a.row_ptr[i];
        v[k] = a.act == DSMP_ACT_RELU ? (yv > 0.0f ? g[k] : 0.0f) : g[k];
      }
    }
    __syncthreads();   // the previous chunk's rows are consumed
#pragma unroll
    for (int k = 0; k < NU; ++k) {
      ys[li + NPW * k][c] = v[k];
      hs[li + NPW * k][c] = hv[k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < NU; ++k) {
      const int64_t i = b + li + NPW * k;
      if (i < i1) {
        const float gm = deg[k] > 0 ? v[k] / (float)deg[k] : 0.0f;
        a.gF[i * DL + c] = gm;
        reinterpret_cast<T*>(a.gT)[i * DL + c] = (T)gm;
      }
    }
    // dh_node = [G] + Wr^T ybar, each output summed over q in order
    float sdh[NU];
#pragma unroll
    for (int k = 0; k < NU; ++k) sdh[k] = a.residual ? g[k] : 0.0f;
#pragma unroll 4
    for (int qq = 0; qq < DL; ++qq) {
      const float w = wr[qq][c];
#pragma unroll
      for (int k = 0; k < NU; ++k) sdh[k] += w * ys[li + NPW * k][qq];
    }
#pragma unroll
    for (int k = 0; k < NU; ++k) {
      const int64_t i = b + li + NPW * k;
      if (i < i1) a.dh_node[i * DL + c] = sdh[k];
    }
    // partial sums of dWr and dbr over the chunk's nodes in order (rows past
    // the end are zero)
    for (int n = 0; n < NB; ++n) {
      const float yv = ys[n][q];
#pragma unroll
      for (int u = 0; u < PP; ++u) acc[u] += yv * hs[n][p0 + u];
      accb += yv;
    }
  }
  float* out = a.p_root + (size_t)blockIdx.x * (DL * DL + DL);
#pragma unroll
  for (int u = 0; u < PP; ++u) out[q * DL + p0 + u] = acc[u];
  if (tid < DL) out[DL * DL + q] = accb;
}

// bf16 layers, d = 64 or 128: the same node terms on matrix cores, with NW
// waves and a step of NR = 32 NW / (d / 32) destinations.  Wave w holds the
// 32 x 32 block (row tile w / QT, column tile w % QT) of the step in the
// accumulator layout
// (lane = column, register r = row 8(r/4) + 4h + r%4), so that every global
// load and store covers whole cache lines across the lanes.  ybar, split into
// bf16 high and low parts (their sum is within 2^-17 of ybar), and h (bf16
// already) go to LDS transposed, [column][row]; from there
//   dh_node = [G] + Wr^T ybar : A = ybar rows (transposing reads), B = Wr
//                               columns (registers; Wr holds bf16 values);
//   dWr += ybar^T h           : A = ybar columns, B = h columns, K = the
//                               step's destinations; each wave keeps
//                               QT*QT/NW tiles of the workgroup's partial sum.
template <int DL, int NW>
struct BNodeShape {
  static constexpr int QT = DL / 32, RT = NW / QT, NR = 32 * RT;  // column tiles, row tiles, rows per step
  static constexpr int TP = NR * 2 + 16 * tr_pad_units(NR * 2);   // LDS pitch of a transposed row (bytes)
  static constexpr int NPAIR = QT * QT / NW;                      // dWr tiles per wave
  static_assert(NPAIR >= 1 && QT * QT % NW == 0, "whole dWr tiles per wave");
};

template <int DL, int NW>
__global__ __launch_bounds__(NW * 64, 8 / NW) void k_bwd_node_m(BNodeArgs a) {
  using M = MT<__bf16>;
  using S = BNodeShape<DL, NW>;
  constexpr int QT = S::QT, NR = S::NR, TP = S::TP, SK = DL / 16, KR = NR / 16;
  __shared__ __align__(16) unsigned char yth[DL * TP], ytl[DL * TP], ht[DL * TP];
  __shared__ float dbs[NW][32];
  const int tid = threadIdx.x, lane = tid & 63, hh = lane >> 5, l32 = lane & 31;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: row bases in scalar registers
  const int rt = wv / QT, ct = wv % QT, q = 32 * ct + l32;
  // B operand of dh_node: lane (p, h) holds Wr[16s + 8h + t][32ct + p]
  bf16x8 bw[SK];
#pragma unroll
  for (int s = 0; s < SK; ++s) {
    float v[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) v[t] = a.wr[(size_t)(16 * s + 8 * hh + t) * DL + q];
    bw[s] = pack_frag<__bf16>(v);   // exact: the values are bf16 already
  }
  f32x16 acc2[S::NPAIR];
#pragma unroll
  for (int j = 0; j < S::NPAIR; ++j) acc2[j] = f32x16{};
  float dbr = 0.0f;
  // Register r of the accumulator layout is row 8(r/4) + 4h + r%4 of the
  // block: a scalar base per row group r/4, one lane byte offset and a
  // constant per register.
  const uint32_t lo4 = (uint32_t)(4 * hh * DL + q) * 4u, lo2 = lo4 / 2;
  auto row_of = [&](int r) { return 8 * (r / 4) + 4 * hh + r % 4; };
  auto at4 = [&](const float* base, int64_t row0, int r) {   // element (row0 + row_of(r), q) of an fp32 array
    return reinterpret_cast<const float*>(reinterpret_cast<const char*>(base + (row0 + 8 * (r / 4)) * DL) + lo4) +
           (r % 4) * DL;
  };
  auto at2 = [&](const __bf16* base, int64_t row0, int r) {
    return reinterpret_cast<const __bf16*>(reinterpret_cast<const char*>(base + (row0 + 8 * (r / 4)) * DL) + lo2) +
           (r % 4) * DL;
  };
  const __bf16* hin = reinterpret_cast<const __bf16*>(a.h_in);
  const int64_t i0 = (int64_t)blockIdx.x * a.per_block;
  const int64_t i1 = i0 + a.per_block < a.n_dst ? i0 + a.per_block : a.n_dst;
  for (int64_t b = i0; b < i1; b += NR) {
    const int64_t rb = b + 32 * rt;   // first row of the wave's block
    const bool full = rb + 32 <= i1;
    float invl;   // lane l32: 1 / degree of row rb + l32 (0 without edges or past the end)
    {
      const int64_t i = rb + l32 < i1 ? rb + l32 : i1 - 1;
      const int32_t d0 = a.row_ptr[i], d1 = a.row_ptr[i + 1];
      const int deg = rb + l32 < i1 ? d1 - d0 : 0;
      invl = deg > 0 ? 1.0f / (float)deg : 0.0f;
    }
    float Y[16], H[16], yb[16];
    if (full) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        yb[r] = *at4(a.G, rb, r);
        Y[r] = *at4(a.y, rb, r);
        H[r] = to_f(*at2(hin, rb, r));
      }
    } else {   // rows past the end re-read the last row
      const int64_t rbl = rb < i1 ? rb : i1 - 1;
      const int rlast = (int)(i1 - 1 - rbl);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t o = (int64_t)(row_of(r) < rlast ? row_of(r) : rlast) * DL + q;
        yb[r] = a.G[rbl * DL + o];
        Y[r] = a.y[rbl * DL + o];
        H[r] = to_f(hin[rbl * DL + o]);
      }
    }
    float gm[16];
    const bool relu = a.act == DSMP_ACT_RELU;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const bool ok = full || rb + row_of(r) < i1;
      const float inv = __shfl(invl, row_of(r), 64);
      const float v = ok && (!relu || Y[r] > 0.0f) ? yb[r] : 0.0f;
      yb[r] = v;
      H[r] = ok ? H[r] : 0.0f;
      dbr += v;
      gm[r] = v * inv;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (full || rb + row_of(r) < i1) {
        *const_cast<float*>(at4(a.gF, rb, r)) = gm[r];
        *const_cast<__bf16*>(at2(reinterpret_cast<const __bf16*>(a.gT), rb, r)) = (__bf16)gm[r];
      }
    __syncthreads();   // the previous step's LDS reads are done
    // transposed rows: [column q][row of the step]
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float vh[4], vl[4], vx[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float y = yb[4 * g + u], yh = (float)(__bf16)y;
        vh[u] = yh;
        vl[u] = y - yh;
        vx[u] = H[4 * g + u];
      }
      const int off = q * TP + (32 * rt + 8 * g + 4 * hh) * 2;
      auto put = [&](unsigned char* base, const float* v) {
        const bf16x2 p0 = __builtin_convertvector((f32x2){v[0], v[1]}, bf16x2);
        const bf16x2 p1 = __builtin_convertvector((f32x2){v[2], v[3]}, bf16x2);
        *reinterpret_cast<uint2*>(base + off) = make_uint2(__builtin_bit_cast(uint32_t, p0), __builtin_bit_cast(uint32_t, p1));
      };
      put(yth, vh);
      put(ytl, vl);
      put(ht, vx);
    }
    __syncthreads();
    // dh_node of the wave's block
    f32x16 C = f32x16{};
#pragma unroll
    for (int s = 0; s < SK; ++s) {
      C = M::mma(lds_frag_rows(yth, TP, 16 * s, 32 * rt), bw[s], C);
      C = M::mma(lds_frag_rows(ytl, TP, 16 * s, 32 * rt), bw[s], C);
    }
    // dh_node = [G] + C, G read again (the step's rows are in the cache)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (full || rb + row_of(r) < i1)
        *const_cast<float*>(at4(a.dh_node, rb, r)) = (a.residual ? *at4(a.G, rb, r) : 0.0f) + C[r];
    // the wave's dWr tiles over the step's rows
#pragma unroll
    for (int j = 0; j < S::NPAIR; ++j) {
      const int idx = wv * S::NPAIR + j, qt = idx / QT, pt = idx % QT;
#pragma unroll
      for (int k = 0; k < KR; ++k) {
        const int co = (16 * k + 8 * hh) * 2;
        const bf16x8 ah = *reinterpret_cast<const bf16x8*>(yth + (32 * qt + l32) * TP + co);
        const bf16x8 al = *reinterpret_cast<const bf16x8*>(ytl + (32 * qt + l32) * TP + co);
        const bf16x8 bh = *reinterpret_cast<const bf16x8*>(ht + (32 * pt + l32) * TP + co);
        acc2[j] = M::mma(ah, bh, acc2[j]);
        acc2[j] = M::mma(al, bh, acc2[j]);
      }
    }
  }
  float* out = a.p_root + (size_t)blockIdx.x * (DL * DL + DL);
#pragma unroll
  for (int j = 0; j < S::NPAIR; ++j) {
    const int idx = wv * S::NPAIR + j, qt = idx / QT, pt = idx % QT;
#pragma unroll
    for (int r = 0; r < 16; ++r) out[(size_t)(32 * qt + 8 * (r / 4) + 4 * hh + r % 4) * DL + 32 * pt + l32] = acc2[j][r];
  }
  // dbr: the two lane halves, then the row tiles of each column tile in order
  dbr += __shfl_xor(dbr, 32, 64);
  if (lane < 32) dbs[wv][lane] = dbr;
  __syncthreads();
  if (tid < DL) {
    float sb = 0.0f;
#pragma unroll
    for (int r = 0; r < S::RT; ++r) sb += dbs[r * QT + tid / 32][tid % 32];
    out[DL * DL + tid] = sb;
  }
}

// db3[p*d+q] = sum_i (sum_{e in E_i} h_{src(e)}[p]) g_i[q] over a chunk of destinations.
template <typename T, int DL>
__global__ __launch_bounds__(256) void k_bwd_db3(int64_t n_dst, int64_t per_block, const int32_t* __restrict__ row_ptr,
                                                 const int32_t* __restrict__ col, const unsigned char* __restrict__ h_in,
                                                 const float* __restrict__ gF, float* __restrict__ part) {
  constexpr int PP = DL * DL / 256, NB = 16;
  __shared__ float hsum[NB][DL];
  __shared__ float gs[NB][DL];
  const T* hin = reinterpret_cast<const T*>(h_in);
  const int p = threadIdx.x % DL, q0 = (threadIdx.x / DL) * PP;
  float acc[PP];
#pragma unroll
  for (int u = 0; u < PP; ++u) acc[u] = 0.0f;
  const int64_t i0 = (int64_t)blockIdx.x * per_block;
  const int64_t i1 = i0 + per_block < n_dst ? i0 + per_block : n_dst;
  for (int64_t b = i0; b < i1; b += NB) {
    __syncthreads();
    for (int u = threadIdx.x; u < NB * DL; u += 256) {
      const int64_t i = b + u / DL;
      const int c = u % DL;
      float s = 0.0f, gv = 0.0f;
      if (i < i1) {
        for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) s += to_f(hin[(int64_t)col[e] * DL + c]);
        gv = gF[i * DL + c];
      }
      hsum[u / DL][c] = s;
      gs[u / DL][c] = gv;
    }
    __syncthreads();
    for (int n = 0; n < NB; ++n) {
      const float hv = hsum[n][p];
#pragma unroll
      for (int u = 0; u < PP; ++u) acc[u] += hv * gs[n][q0 + u];
    }
  }
  float* out = part + (size_t)blockIdx.x * DL * DL;
#pragma unroll
  for (int u = 0; u < PP; ++u) out[p * DL + q0 + u] = acc[u];
}

// ------------------------------------------------------------ dz kernel

struct DzArgs {
  int64_t E;
  const int32_t* col;
  const int32_t* dst;
  const unsigned char* h_in;   // [n_src][d]
  const float* gF;             // [n_dst][d] fp32
  const unsigned char* packed;
  PackLayout L;
  const unsigned char* zE;     // [E][h2] permuted order
  const unsigned char* zmask;  // [E][(h1+h2)/8] ReLU mask bits of z1 and z (forward)
  unsigned char* da2E;         // [E][h2] permuted order, layer dtype
  unsigned char* da1E;         // [E][h1] permuted order, layer dtype
  const unsigned char* U;      // aggregate form: [n_dst][h2][d] layer dtype, U_i[k][p]
  const unsigned char* gT;     // aggregate form: g_i [n_dst][d] layer dtype
  int64_t n_dst;
  const int32_t* row_ptr;      // aggregate form: edges of each destination
  int nb;                      // k_bwd_dz_agg: destinations per block, 1 .. DZ_NB (0: DZ_NB)
};

template <typename T, int DL, int H1, int H2>
struct DzShape {
  static constexpr int KS = MT<T>::KS, EPL = MT<T>::EPL;
  static constexpr int NT = (H2 <= 64 || (H2 <= 128 && sizeof(T) == 2)) ? 2 : 1, TILE = 4 * NT * 32;
  static constexpr int KT = H2 / 32, JT = H1 / 32, SKD = DL / KS, SK2 = H2 / KS;
  static constexpr int ESZ = sizeof(T);
  static constexpr int ROWB = DL * ESZ + 16;
  static constexpr int RCH = (H2 * DL * ESZ <= 32768) ? H2 : 32768 / (DL * ESZ);
  static constexpr int CPP = H2 / RCH, KPC = RCH / 32, NCH = DL * CPP;
  static constexpr int STAGE = RCH * ROWB, HROWB = DL * ESZ + 16;
  static constexpr int LDS = 2 * STAGE + TILE * HROWB;
};

// Epilogue of the dz kernels: acc[t][kt] holds dz of the lane's edge (tile t)
// for k in tile kt (register i is permuted position 16*kt + i).  Writes
// da2 = dz * [z > 0] (permuted order), then dz1 = W2^T da2 on MFMA and
// da1 = dz1 * [z1 > 0].  w2t: W2^T rows [h1][h2 permuted] with a row pitch of
// W2P bytes (the packed copy in global memory, or a copy in LDS).
template <typename T, int DL, int H1, int H2, int NT, int KT, int W2P = H2 * (int)sizeof(T)>
__device__ __forceinline__ void dz_finish(const DzArgs& a, const f32x16 (&acc)[NT][KT], const int64_t (&eid)[NT],
                                          const bool (&valid)[NT], int hh, const unsigned char* w2t) {
  using S = DzShape<T, DL, H1, H2>;
  using M = MT<T>;
  using frag = typename M::frag;
  constexpr int KS = S::KS, EPL = S::EPL, ESZ = S::ESZ;
  const int l32 = threadIdx.x & 31;
  constexpr int MW1 = H1 / 64, MW2 = H2 / 64;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const size_t e = valid[t] ? (size_t)eid[t] : 0;
    // the lane's mask bits: bit b of its half <-> position (b/EPL)*KS + hh*EPL + b%EPL
    uint32_t m1[MW1], m2[MW2];
    {
      const uint32_t* mb = reinterpret_cast<const uint32_t*>(a.zmask + e * ((H1 + H2) / 8));
#pragma unroll
      for (int w = 0; w < MW1; ++w) m1[w] = mb[hh * MW1 + w];
#pragma unroll
      for (int w = 0; w < MW2; ++w) m2[w] = mb[2 * MW1 + hh * MW2 + w];
    }
    frag da2B[S::SK2];
#pragma unroll
    for (int s = 0; s < S::SK2; ++s) {
      float v[EPL];
#pragma unroll
      for (int u = 0; u < EPL; ++u) {
        const int n = s * EPL + u;
        v[u] = keep_if_bit(acc[t][n / 16][n % 16], m2[n / 32], n % 32);
      }
      da2B[s] = pack_frag<T>(v);
      if (valid[t]) *reinterpret_cast<frag*>(a.da2E + (e * H2 + s * KS + hh * EPL) * ESZ) = da2B[s];
    }
#pragma unroll
    for (int jt = 0; jt < S::JT; ++jt) {
      // from LDS the W2^T fragments are cheap to fetch per tile: keep the
      // scheduler from hoisting all of them (registers)
      if constexpr (W2P != H2 * (int)sizeof(T)) __builtin_amdgcn_sched_barrier(0);
      f32x16 C = f32x16{};
#pragma unroll
      for (int s = 0; s < S::SK2; ++s) {
        frag A = ld_frag<T>(w2t + (size_t)(jt * 32 + l32) * W2P + (s * KS + hh * EPL) * ESZ);
        C = M::mma(A, da2B[s], C);
      }
      // register i of tile jt is permuted position n = 16*jt + i
#pragma unroll
      for (int i = 0; i < 16; i += EPL) {
        const int n = 16 * jt + i;
        const int pos = (n / EPL) * KS + hh * EPL;
        float v[EPL];
#pragma unroll
        for (int u = 0; u < EPL; ++u) v[u] = keep_if_bit(C[i + u], m1[(n + u) / 32], (n + u) % 32);
        if (valid[t]) *reinterpret_cast<frag*>(a.da1E + (e * H1 + pos) * ESZ) = pack_frag<T>(v);
      }
    }
  }
}

// dz_e[k] = sum_p h_j[p] sum_q W3[p*d+q][k] g_e[q], accumulated as
// sum_p W3T[p] (h_j[p] g_e): the scale is folded into the B operand, so the
// accumulators are touched only by MFMA and the next p's operand is formed
// while the current products run.
template <typename T, int DL, int H1, int H2>
__global__ __launch_bounds__(256, (DL <= 64 && H2 * sizeof(T) <= 256) ? 2 : 1) void k_bwd_dz(DzArgs a) {
  using S = DzShape<T, DL, H1, H2>;
  using M = MT<T>;
  using frag = typename M::frag;
  constexpr int KS = S::KS, EPL = S::EPL, NT = S::NT, TILE = S::TILE, ESZ = S::ESZ;
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* stage0 = smem;
  unsigned char* htile = smem + 2 * S::STAGE;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  const int64_t t0 = (int64_t)blockIdx.x * TILE;
  const unsigned char* P = a.packed;

  int64_t eid[NT];
  int dnode[NT], hrow[NT];
  bool valid[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    hrow[t] = (wv * NT + t) * 32 + l32;
    eid[t] = t0 + hrow[t];
    valid[t] = eid[t] < a.E;
    dnode[t] = valid[t] ? a.dst[eid[t]] : 0;
  }
  {
    constexpr int HU = DL * ESZ / 16;
    for (int u = tid; u < TILE * HU; u += 256) {
      int r = u / HU, c = u % HU;
      int64_t e = t0 + r;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (e < a.E) v = reinterpret_cast<const uint4*>(a.h_in + (size_t)a.col[e] * DL * ESZ)[c];
      *reinterpret_cast<uint4*>(htile + r * S::HROWB + c * 16) = v;
    }
  }
  // the lane's g_e values (its half of every K step), fp32
  float gv[NT][S::SKD][EPL];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int s = 0; s < S::SKD; ++s)
#pragma unroll
      for (int u = 0; u < EPL; ++u) gv[t][s][u] = a.gF[(size_t)dnode[t] * DL + s * KS + hh * EPL + u];

  f32x16 acc[NT][S::KT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int kt = 0; kt < S::KT; ++kt) acc[t][kt] = f32x16{};

  const unsigned char* A3 = P + a.L.w3t;   // [p][k][q]
  // W3T chunks go straight into LDS, one chunk ahead of the products
  using St = LdsStage<S::RCH, DL * ESZ>;
  static_assert(St::BYTES == S::STAGE, "stage layout");
  St stg;
  stg.init();
  auto chunk = [&](int c) {
    return A3 + ((size_t)(c / S::CPP) * H2 + (size_t)(c % S::CPP) * S::RCH) * DL * ESZ;
  };
  stg.issue(chunk(0), stage0);
  stage_wait();
  __syncthreads();
  // scaled B operand for p = 0
  frag Bq[NT][S::SKD];
  auto form = [&](int p, frag (&B)[NT][S::SKD]) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const float sc = to_f(*reinterpret_cast<const T*>(htile + hrow[t] * S::HROWB + p * ESZ));
#pragma unroll
      for (int s = 0; s < S::SKD; ++s) {
        float v[EPL];
#pragma unroll
        for (int u = 0; u < EPL; ++u) v[u] = sc * gv[t][s][u];
        B[t][s] = pack_frag<T>(v);
      }
    }
  };
  // Products of W3T[p] (chunk by chunk) against Bq; once a fragment Bq[t][s]
  // has fed its last product of this p it is re-formed in place for p+1, so
  // the formation overlaps the remaining products.
  form(0, Bq);
  for (int p = 0; p < DL; ++p) {
    float scn[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
      scn[t] = p + 1 < DL ? to_f(*reinterpret_cast<const T*>(htile + hrow[t] * S::HROWB + (p + 1) * ESZ)) : 0.0f;
#pragma unroll
    for (int cc = 0; cc < S::CPP; ++cc) {
      const int c = p * S::CPP + cc;
      const int buf = c & 1;
      if (c + 1 < S::NCH) stg.issue(chunk(c + 1), stage0 + (buf ^ 1) * S::STAGE);
      const unsigned char* sb = stage0 + buf * S::STAGE;
#pragma unroll
      for (int s = 0; s < S::SKD; ++s) {
#pragma unroll
        for (int kq = 0; kq < S::KPC; ++kq) {
          frag A = ld_frag<T>(sb + (kq * 32 + l32) * S::ROWB + (s * KS + hh * EPL) * ESZ);
#pragma unroll
          for (int t = 0; t < NT; ++t) acc[t][cc * S::KPC + kq] = M::mma(A, Bq[t][s], acc[t][cc * S::KPC + kq]);
        }
        if (cc == S::CPP - 1) {
#pragma unroll
          for (int t = 0; t < NT; ++t) {
            float v[EPL];
#pragma unroll
            for (int u = 0; u < EPL; ++u) v[u] = scn[t] * gv[t][s][u];
            Bq[t][s] = pack_frag<T>(v);
          }
        }
      }
      stage_wait();
      __syncthreads();
    }
  }

  dz_finish<T, DL, H1, H2, NT, S::KT>(a, acc, eid, valid, hh, a.packed + a.L.w2t);
}

// Aggregate form of dz.  With U_i[k][p] = sum_q W3[p*d+q][k] g_i[q] for
// every destination (one GEMM, k_u_gemm), dz_e[k] = sum_p U_i[k][p] h_j[p]
// for each edge e into i.  The work items are 32-edge tiles of one
// destination: the A operand is U_i^T, the B operand the lane's own gathered
// row h_j (zero past the destination's last edge).  Workgroups are persistent
// (as many as fit on the device), so W2^T of the epilogue is copied to LDS
// once per workgroup; each takes blocks of DZ_NB consecutive destinations in
// turn and lists their tiles in LDS, and its four waves take consecutive
// tiles, so the tiles of one destination run side by side and U_i comes from
// HBM once.
constexpr int DZ_NB = 16;

template <typename T, int H1, int H2>
struct DzAggShape {
  static constexpr int W2P = H2 * (int)sizeof(T) + 16;   // LDS row pitch of W2^T
  static constexpr int LDS = H1 * W2P;
};

template <typename T, int DL, int H1, int H2>
__global__ __launch_bounds__(256, (DL <= 64 && H2 * sizeof(T) <= 256) ? 3 : 1) void k_bwd_dz_agg(DzArgs a) {
  using S = DzShape<T, DL, H1, H2>;
  using SA = DzAggShape<T, H1, H2>;
  using M = MT<T>;
  using frag = typename M::frag;
  constexpr int KS = S::KS, EPL = S::EPL, ESZ = S::ESZ, KT = S::KT, SKD = S::SKD, NT = 1;
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  {
    LdsStage<H1, H2 * ESZ> stg;
    stg.init();
    stg.issue(a.packed + a.L.w2t, smem);
    stage_wait();
    __syncthreads();
  }
  __shared__ int tstart[DZ_NB + 1];   // first tile of each destination of the block
  const int NB = a.nb > 0 && a.nb < DZ_NB ? a.nb : DZ_NB;
  const int64_t nblk = (a.n_dst + NB - 1) / NB;
  for (int64_t blk = blockIdx.x; blk < nblk; blk += gridDim.x) {
    const int64_t d0 = blk * NB;
    const int nd = (int)(a.n_dst - d0 < NB ? a.n_dst - d0 : NB);
    if (wv == 0) {
      // tiles per destination, inclusive prefix over the block's lanes
      int nt = 0;
      if (lane < nd) nt = (a.row_ptr[d0 + lane + 1] - a.row_ptr[d0 + lane] + 31) / 32;
#pragma unroll
      for (int o = 1; o < DZ_NB; o <<= 1) {
        const int v = __shfl_up(nt, o, 64);
        if (lane >= o) nt += v;
      }
      if (lane < DZ_NB) tstart[lane + 1] = nt;
      if (lane == 0) tstart[0] = 0;
    }
    __syncthreads();
    const int ntile = tstart[nd];
    for (int tau = wv; tau < ntile; tau += 4) {
      int k = 0;
      while (tstart[k + 1] <= tau) ++k;   // destination of tile tau (k < nd)
      const int64_t i = d0 + k;
      const int64_t pa = a.row_ptr[i], pb = a.row_ptr[i + 1];
      const int64_t c0 = pa + (int64_t)(tau - tstart[k]) * 32;
      // U_i in fragment order: fragment (kt, s) is 64 lanes x EPL elements
      const unsigned char* ur = a.U + ((size_t)i * H2 * DL + lane * EPL) * ESZ;
      int64_t eid[NT];
      bool valid[NT];
      frag hB[NT][SKD];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        eid[t] = c0 + t * 32 + l32;
        valid[t] = eid[t] < pb;
        const unsigned char* hr = a.h_in + (size_t)(valid[t] ? a.col[eid[t]] : 0) * DL * ESZ;
#pragma unroll
        for (int s = 0; s < SKD; ++s) hB[t][s] = valid[t] ? ld_frag<T>(hr + (s * KS + hh * EPL) * ESZ) : frag{};
      }
      f32x16 acc[NT][KT];
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) {
        frag A[SKD];
#pragma unroll
        for (int s = 0; s < SKD; ++s) A[s] = ld_frag<T>(ur + (size_t)((kt * SKD + s) * 64 * EPL) * ESZ);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          acc[t][kt] = f32x16{};
#pragma unroll
          for (int s = 0; s < SKD; ++s) acc[t][kt] = M::mma(A[s], hB[t][s], acc[t][kt]);
        }
      }
      dz_finish<T, DL, H1, H2, NT, KT, SA::W2P>(a, acc, eid, valid, hh, smem);
    }
    __syncthreads();   // the block's tile list is read until every wave is done
  }
}

// Fused edge gradients of the aggregate form (bf16 layers, h1 = h2 <= 128).
// One pass over 32-edge tiles computes dz = U_i h_j, the masked da2,
// dz1 = W2^T da2 and da1 (as k_bwd_dz_agg does), and folds the per-edge
// weight gradients straight into per-workgroup sums, so da2 and da1 never go
// to HBM.  A workgroup takes blocks of 16 destinations; a tile is 32
// consecutive edges of the block's rows, so it may cross destinations: dz
// runs once per destination in the tile, with the B operand restricted to
// that destination's lanes (every tile is full but the block's last, where a
// tile per destination would leave most tails part-empty).  The sums:
//   dW2[k][j] = sum_e da2_e[k] z1_e[j],  db2 = sum_e da2_e,
//   dW1[j][c] = sum_e da1_e[j] x_e[c],   db1 = sum_e da1_e.
// A workgroup of eight waves takes four tiles per round; the two waves of a
// pair share one tile and its LDS slot (dz split by k tiles, dz1 by j tiles,
// the z1 row by halves).  The slot receives the tile's rows of da2, da1 and
// z1 and its split attributes.  z1 = ReLU(W1 x + b1) is recomputed on the
// matrix cores from bf16 high and low parts, W1h xh + W1h xl + W1l xh + b1h
// + b1l with fp32 accumulation: within about 2^-16 of the forward's fp32
// value, far inside the bf16 rounding that z1 and da2 then take, and a ReLU
// decision can only differ where z1 is about zero.  The attributes enter dW1
// the same way (high parts in columns 0..7, low parts in 8..15) next to a
// column of ones (16) that gives db1; db2 sums the da2 fragments of the
// products.  After a barrier the four slots are contracted over their edges
// with transposing LDS reads, each wave taking its share of the dW2 tiles.
// Each load of the wave's next tile goes out as soon as its registers are
// free (its source index one round earlier still), so they are in flight
// while the products run; the barriers order LDS traffic only.
// Partial sums go to slot blockIdx.x of the dW2/db2 and dW1/db1 partial
// buffers, summed later in a fixed order.
struct EdgeGradArgs {
  DzArgs dz;
  const float* node_attr;
  int dim, attr_mode, de;
  unsigned char* da1_out;   // [E][h1] bf16 permuted order, or null (needed for the attribute gradient)
  float* p_w2;              // [gridDim.x][h2*h1 + h2]
  float* p_w1;              // [gridDim.x][h1*de + h1]
};

template <int DL, int H1, int H2>
struct EdgeGradShape {
  static_assert(H1 == H2 && (H1 == 64 || H1 == 128), "fused edge gradients: h1 = h2 = 64 or 128");
  static constexpr int NW = 8, NT = NW * 64;                    // waves, threads
  static constexpr int W2P = H2 * 2 + 16;                       // LDS pitch of W2^T rows
  // LDS pitches of the slot rows: four consecutive rows of a transposing read
  // land 8 banks apart (pitch = 8 dwords mod 64), so its 16-lane groups are
  // free of bank conflicts
  static constexpr int DA2P = H2 * 2 + 32, DA1P = H1 * 2 + 32;  // da2 / da1 / z1 rows
  static constexpr int XSP = 96;                                // 32 bf16 attribute columns
  static constexpr int OD1 = 32 * DA2P, OZ1 = OD1 + 32 * DA1P, OXS = OZ1 + 32 * DA1P;
  static constexpr int SLOT = OXS + 32 * XSP;
  static constexpr int W2B = H1 * W2P, W1B = H1 * 9 * 4;
  static constexpr int LDS = W2B + W1B + 4 * SLOT;
  static_assert(LDS <= 160 * 1024 - 256, "LDS of the fused edge-gradient kernel");
  static constexpr int KT = H2 / 32, JT = H1 / 32;
  static constexpr int TPW = KT * JT >= NW ? KT * JT / NW : 1;   // dW2 tiles per wave
  static constexpr int ACTIVE = KT * JT / TPW;                     // waves with dW2 tiles
};

template <int DL, int H1, int H2>
__global__ __launch_bounds__(512, 1) void k_bwd_edge_agg(EdgeGradArgs g) {
  using S = DzShape<__bf16, DL, H1, H2>;
  using G = EdgeGradShape<DL, H1, H2>;
  using M = MT<__bf16>;
  using frag = bf16x8;
  constexpr int KS = S::KS, EPL = S::EPL, KT = S::KT, SKD = S::SKD, SK2 = S::SK2, JT = S::JT;
  constexpr int SK1 = H1 / KS, MW1 = H1 / 64, MW2 = H2 / 64;
  constexpr int KTH = KT / 2, JTH = JT / 2, SK1H = SK1 / 2, SK2H = SK2 / 2;   // per half of a pair
  constexpr int ZB = SK1H / 2;   // 32-row blocks of z1 per half
  const DzArgs& a = g.dz;
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* w2s = smem;
  float* w1s = reinterpret_cast<float*>(smem + G::W2B);   // [H1][8] lane order, then b1 [H1]
  unsigned char* slots = smem + G::W2B + G::W1B;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  const int pr = wv & 3, hf = wv >> 2;   // tile (slot) of the wave's pair, half of the pair
  if (tid < 256) {   // the staging helpers are written for 256 threads
    LdsStage<H1, H2 * 2> stg;
    stg.init();
    stg.issue(a.packed + a.L.w2t, w2s);
    lds_copy_async(a.packed + a.L.w1l, reinterpret_cast<unsigned char*>(w1s), H1 * 8 * 4 / 16);
    lds_copy_async(a.packed + a.L.b1l, reinterpret_cast<unsigned char*>(w1s + H1 * 8), H1 * 4 / 16);
  }
  // products: dW2 tiles (kt(m), jt) of this wave, db2 of kt(m) where kt(m) % JT == jt
  const int jt = wv % JT;
  const bool active = wv < G::ACTIVE;
  auto kt_of = [&](int m) { return (wv / JT) * G::TPW + m; };
  f32x16 acc2[G::TPW], acc1 = f32x16{};
#pragma unroll
  for (int m = 0; m < G::TPW; ++m) acc2[m] = f32x16{};
  int bm = -1;   // the tile m whose db2 this wave forms
#pragma unroll
  for (int m = 0; m < G::TPW; ++m)
    if (active && kt_of(m) % JT == jt) bm = m;
  float db2 = 0.0f;   // the lane's half of the edges, column kt(bm)*32 + l32
  stage_wait();
  __syncthreads();   // W2^T and the layer-1 weights are in LDS

  __shared__ int rps[DZ_NB + 1];
  __shared__ int slot_cnt[4];
  unsigned char* myslot = slots + pr * G::SLOT;
  // A operands of the z1 product, built each round from the fp32 weights in
  // LDS: row R of block zb holds the layer-1 weights of stored position
  // (hf*SK1H + 2zb + i/8)*16 + hh'*8 + i%8 with R = 8(i/4) + 4hh' + i%4; K
  // slots 0..7 W1h, 8..15 W1h, 16..23 W1l, 24 b1h, 25 b1l
  auto w1_frags = [&](int zb, frag& f0, frag& f1) {
    const int R = l32, i = 4 * (R / 8) + R % 4, hr = (R % 8) / 4;
    const int pos = (hf * SK1H + 2 * zb + i / 8) * KS + hr * EPL + i % 8;
    const int hn = ((pos % KS) / EPL) * (H1 / 2) + (pos / KS) * EPL + pos % EPL;
    const f32x4 wa = *reinterpret_cast<const f32x4*>(w1s + hn * 8);
    const f32x4 wb = *reinterpret_cast<const f32x4*>(w1s + hn * 8 + 4);
    const float wv[8] = {wa[0], wa[1], wa[2], wa[3], wb[0], wb[1], wb[2], wb[3]};
    const float bb = w1s[H1 * 8 + hn];
    float v0[8], v1[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const float whi = (float)(__bf16)wv[c];
      v0[c] = whi;                        // slots 0..7 (times xh) and 8..15 (times xl)
      v1[c] = hh ? 0.0f : wv[c] - whi;    // slots 16..23 (times xh)
    }
    if (hh) {
      const float bhi = (float)(__bf16)bb;
      v1[0] = bhi;
      v1[1] = bb - bhi;
    }
    f0 = pack_frag<__bf16>(v0);
    f1 = pack_frag<__bf16>(v1);
  };

  // a tile of the current block: 32 consecutive edges of the block's edge
  // range (destinations d0 .. d0 + nd - 1, rows in order), which may span
  // several destinations: the first and last of them, the first edge, the
  // lane's edge, its source and its destination
  struct Tile {
    int i0, i1, c0, eid, cnt, jn, dn;   // graph indices are int32
    bool has, valid;
  };
  // the operands of a tile: gathered row, the half's rows of U_i, mask bits, node attribute rows
  struct Ops {
    frag hB[SKD], UA[KTH][SKD];
    uint32_t m1[MW1], m2[MW2];
    float ri[4], rj[4];
  };
  int d0 = 0;
  int ntile = 0;
  int nd = 0;
  auto locate = [&](int tau, Tile& t) {
    t.has = tau < ntile;
    t.i0 = t.i1 = d0; t.c0 = 0; t.eid = 0; t.cnt = 0; t.valid = false;
    if (!t.has) return;
    const int pe = rps[nd];
    t.c0 = rps[0] + tau * 32;
    t.eid = t.c0 + l32;
    t.valid = t.eid < pe;
    t.cnt = pe - t.c0 < 32 ? pe - t.c0 : 32;
    // destination of an edge of the block: the number of row ends at or below it
    const int re = lane < nd ? rps[lane + 1] : 0x7fffffff;
    t.i0 = d0 + __popcll(__ballot(re <= t.c0));
    t.i1 = d0 + __popcll(__ballot(re <= t.c0 + t.cnt - 1));
  };
  // Loads are unconditional (lanes past the tile read edge 0) so that no
  // select waits on them; the dz part zeroes those lanes.
  auto load_col = [&](Tile& t) {
    const int e = t.valid ? t.eid : 0;
    t.jn = a.col[e];
    t.dn = a.dst[e];
  };
  // the gathered row and the half's rows of U_i (issued as soon as the
  // previous tile's products have read those registers) ...
  auto load_uh = [&](const Tile& t, Ops& o) {
    if (!t.has) return;
    const int i = __builtin_amdgcn_readfirstlane(t.i0);   // the tile's first destination
    const unsigned char* ub = a.U + (size_t)i * (H2 * DL * 2);   // fragment order
    const unsigned char* hr = a.h_in + (size_t)t.jn * DL * 2;
#pragma unroll
    for (int s = 0; s < SKD; ++s) o.hB[s] = ld_frag<__bf16>(hr + (s * KS + hh * EPL) * 2);
#pragma unroll
    for (int q = 0; q < KTH; ++q)
#pragma unroll
      for (int s = 0; s < SKD; ++s)
        o.UA[q][s] = ld_frag<__bf16>(ub + (uint32_t)((((hf * KTH + q) * SKD + s) * 64 + lane) * EPL * 2));
  };
  // ... the node attribute rows and z's mask bits (after their use in the
  // first step) and z1's mask bits (after the second step); each load goes
  // out once its registers are free
  auto load_attr = [&](const Tile& t, Ops& o) {
    if (!t.has) return;
    const int nw = g.dim + 1;
    const float* vi = g.node_attr + (size_t)t.dn * nw;
    const float* vj = g.node_attr + (size_t)t.jn * nw;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int cc = c < nw ? c : nw - 1;   // in the row; unused past dim
      o.ri[c] = vi[cc];
      o.rj[c] = vj[cc];
    }
  };
  auto load_m2 = [&](const Tile& t, Ops& o) {
    if (!t.has) return;
    const size_t e = t.valid ? (size_t)t.eid : 0;
    const uint32_t* mb = reinterpret_cast<const uint32_t*>(a.zmask + e * ((H1 + H2) / 8));
#pragma unroll
    for (int w = 0; w < MW2; ++w) o.m2[w] = mb[2 * MW1 + hh * MW2 + w];
  };
  auto load_m1 = [&](const Tile& t, Ops& o) {
    if (!t.has) return;
    const size_t e = t.valid ? (size_t)t.eid : 0;
    const uint32_t* mb = reinterpret_cast<const uint32_t*>(a.zmask + e * ((H1 + H2) / 8));
#pragma unroll
    for (int w = 0; w < MW1; ++w) o.m1[w] = mb[hh * MW1 + w];
  };

  // ---- dz part, first step: the half's k tiles of dz, its da2 columns, z1
  // columns and (half 0) the split attribute row go into the pair's slot
  frag da2B[SK2];
  auto dz_part1 = [&](auto half, const Tile& t, const Tile& nxt, Ops& o) {
    constexpr int hf = decltype(half)::value;
    float x[8];
    edge_attr_rows(o.ri, o.rj, g.dim, g.attr_mode, x);
#pragma unroll
    for (int c = 0; c < 8; ++c) x[c] = t.valid ? x[c] : 0.0f;
    float xh[8], xl[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      xh[c] = (float)(__bf16)x[c];
      xl[c] = x[c] - xh[c];
    }
    // z1 of the half's 32-row blocks on MFMA: B = [xh | xl | xh | 1 1 0..]
    // (lane = edge), A = the rows prepared in w1A; rows of block zb are the
    // stored positions of z1 frags s = hf*SK1H + 2zb + i/8 (half hh, element i%8)
    {
      frag xb0, xb1;
      float v0[8], v1[8];
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        v0[c] = hh ? xl[c] : xh[c];
        v1[c] = hh ? (c < 2 ? 1.0f : 0.0f) : xh[c];
      }
      xb0 = pack_frag<__bf16>(v0);
      xb1 = pack_frag<__bf16>(v1);
      unsigned char* zrow = myslot + G::OZ1 + l32 * G::DA1P;
#pragma unroll
      for (int zb = 0; zb < ZB; ++zb) {
        frag w0, w1;
        w1_frags(zb, w0, w1);
        f32x16 Z = f32x16{};
        Z = M::mma(w0, xb0, Z);
        Z = M::mma(w1, xb1, Z);
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int s = hf * SK1H + 2 * zb + q;
          float zv[EPL];
#pragma unroll
          for (int u = 0; u < EPL; ++u) zv[u] = relu_bits(Z[8 * q + u]);
          *reinterpret_cast<frag*>(zrow + (s * KS + hh * EPL) * 2) = pack_frag<__bf16>(zv);
        }
      }
    }
    if (hf == 0) {
      // columns 16hh .. 16hh+15: high parts (0..7), low parts (8..15), ones (16), zeros
      float xv[16];
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        xv[c] = hh ? (c == 0 && t.valid ? 1.0f : 0.0f) : xh[c];
        xv[8 + c] = hh ? 0.0f : xl[c];
      }
      unsigned char* xrow = myslot + G::OXS + l32 * G::XSP + hh * 32;
      *reinterpret_cast<frag*>(xrow) = pack_frag<__bf16>(xv);
      *reinterpret_cast<frag*>(xrow + 16) = pack_frag<__bf16>(xv + 8);
      if (lane == 0) slot_cnt[pr] = t.cnt;
    }
    load_attr(nxt, o);   // the attribute rows have been used
#pragma unroll
    for (int s = 0; s < SKD; ++s)
      if (!t.valid) o.hB[s] = frag{};
    // dz = U_i h_j, one destination of the tile at a time: the B operand
    // keeps the lanes whose edge goes into that destination (U of the first
    // one was loaded a round ahead, the others are loaded here)
    f32x16 acc[KTH];
#pragma unroll
    for (int q = 0; q < KTH; ++q) acc[q] = f32x16{};
    for (int i = t.i0; i <= t.i1; ++i) {
      const bool mine = t.dn == i;
      if (__ballot(mine) == 0) continue;   // a destination without edges
      if (i != t.i0) {
        // a scalar row base and 32-bit lane offsets
        const unsigned char* ub = a.U + (size_t)__builtin_amdgcn_readfirstlane(i) * (H2 * DL * 2);
#pragma unroll
        for (int q = 0; q < KTH; ++q)
#pragma unroll
          for (int s = 0; s < SKD; ++s)
            o.UA[q][s] = ld_frag<__bf16>(ub + (uint32_t)((((hf * KTH + q) * SKD + s) * 64 + lane) * EPL * 2));
      }
      frag hBm[SKD];
#pragma unroll
      for (int s = 0; s < SKD; ++s) hBm[s] = mine ? o.hB[s] : frag{};
#pragma unroll
      for (int q = 0; q < KTH; ++q)
#pragma unroll
        for (int s = 0; s < SKD; ++s) acc[q] = M::mma(o.UA[q][s], hBm[s], acc[q]);
    }
    load_uh(nxt, o);   // the products above have read these registers
    // da2 = dz [z > 0] for the half's positions n = 16 kt + i (frags s = n / EPL)
    unsigned char* d2row = myslot + l32 * G::DA2P;
#pragma unroll
    for (int q = 0; q < SK2H; ++q) {
      const int s = hf * SK2H + q;
      float v[EPL];
#pragma unroll
      for (int u = 0; u < EPL; ++u) {
        const int n = s * EPL + u;
        v[u] = keep_if_bit(acc[n / 16 - hf * KTH][n % 16], o.m2[n / 32], n % 32);
      }
      da2B[s] = pack_frag<__bf16>(v);
      *reinterpret_cast<frag*>(d2row + (s * KS + hh * EPL) * 2) = da2B[s];
    }
    load_m2(nxt, o);   // z's mask bits have been used
  };
  // ---- dz part, second step (da2 of the whole tile is in the slot): the
  // half's j tiles of dz1 = W2^T da2 and da1 = dz1 [z1 > 0]
  auto dz_part2 = [&](auto half, const Tile& t, const Tile& nxt, Ops& o) {
    constexpr int hf = decltype(half)::value;
    const unsigned char* d2row = myslot + l32 * G::DA2P;
#pragma unroll
    for (int q = 0; q < SK2H; ++q) {
      const int s = (1 - hf) * SK2H + q;
      da2B[s] = *reinterpret_cast<const frag*>(d2row + (s * KS + hh * EPL) * 2);
    }
    unsigned char* d1row = myslot + G::OD1 + l32 * G::DA1P;
    const size_t e = t.valid ? (size_t)t.eid : 0;
#pragma unroll
    for (int q = 0; q < JTH; ++q) {
      const int t1 = hf * JTH + q;
      f32x16 C = f32x16{};
#pragma unroll
      for (int s = 0; s < SK2; ++s) {
        frag A = ld_frag<__bf16>(w2s + (size_t)(t1 * 32 + l32) * G::W2P + (s * KS + hh * EPL) * 2);
        C = M::mma(A, da2B[s], C);
      }
#pragma unroll
      for (int i0 = 0; i0 < 16; i0 += EPL) {
        const int n = 16 * t1 + i0;
        const int pos = (n / EPL) * KS + hh * EPL;
        float v[EPL];
#pragma unroll
        for (int u = 0; u < EPL; ++u) v[u] = keep_if_bit(C[i0 + u], o.m1[(n + u) / 32], (n + u) % 32);
        const frag f = pack_frag<__bf16>(v);
        *reinterpret_cast<frag*>(d1row + pos * 2) = f;
        if (g.da1_out && t.valid) *reinterpret_cast<frag*>(g.da1_out + (e * H1 + pos) * 2) = f;
      }
    }
    load_m1(nxt, o);   // z1's mask bits have been used
  };

  // ---- products over a round's slots
  auto products = [&](int nslot) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      if (v < nslot) {
        // The slot's LDS address (past 64 KB, beyond an instruction's offset
        // field) is formed here from a scalar base, not kept per lane and
        // region for the whole kernel: that took a register per slot and
        // region and pushed other values out to scratch.
        uint32_t sb = (uint32_t)(uintptr_t)(slots + v * G::SLOT);
        asm volatile("" : "+s"(sb));
        lds_cu8* st = (lds_cu8*)(uintptr_t)sb;
        const int cnt = slot_cnt[v];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          if (ks * 16 < cnt) {
            if (active) {
              const frag Bz = lds_frag_rows(st + G::OZ1, G::DA1P, 16 * ks, 32 * jt);
              frag A[G::TPW];
#pragma unroll
              for (int m = 0; m < G::TPW; ++m) A[m] = lds_frag_rows(st, G::DA2P, 16 * ks, 32 * kt_of(m));
#pragma unroll
              for (int m = 0; m < G::TPW; ++m) {
                acc2[m] = M::mma(A[m], Bz, acc2[m]);
                if (m == bm) {
#pragma unroll
                  for (int t = 0; t < 8; ++t) db2 += (float)A[m][t];
                }
              }
            }
            if (wv < JT) {
              const frag A1 = lds_frag_rows(st + G::OD1, G::DA1P, 16 * ks, 32 * jt);
              const frag Bx = lds_frag_rows(st + G::OXS, G::XSP, 16 * ks, 0);
              acc1 = M::mma(A1, Bx, acc1);
            }
          }
        }
      }
    }
  };

  // One round: the pair contracts its tile into the slot (two steps around
  // an LDS barrier).  The next round's operands go out into the same
  // registers as soon as they are free (its source index came a round
  // earlier), the tile two rounds ahead takes the place of `cur` and its
  // source index goes out; then the round's slots are contracted while
  // those loads are in flight.
  Ops op;
  auto round = [&](int r0, Tile& cur, const Tile& nxt) {
    if (cur.has) {
      if (hf == 0) dz_part1(std::integral_constant<int, 0>{}, cur, nxt, op);
      else dz_part1(std::integral_constant<int, 1>{}, cur, nxt, op);
    } else {
      load_attr(nxt, op);
      load_uh(nxt, op);
      load_m2(nxt, op);
    }
    lds_barrier();   // the pairs' da2 rows are complete
    if (cur.has) {
      if (hf == 0) dz_part2(std::integral_constant<int, 0>{}, cur, nxt, op);
      else dz_part2(std::integral_constant<int, 1>{}, cur, nxt, op);
    } else {
      load_m1(nxt, op);
    }
    locate(r0 + 8 + pr, cur);
    load_col(cur);
    lds_barrier();   // the round's slots are complete
    products(ntile - r0 < 4 ? ntile - r0 : 4);
    lds_barrier();   // slots are free for the next round
  };

  const int64_t nblk = (a.n_dst + DZ_NB - 1) / DZ_NB;
  for (int64_t blk = blockIdx.x; blk < nblk; blk += gridDim.x) {
    d0 = (int)(blk * DZ_NB);
    nd = (int)(a.n_dst - d0 < DZ_NB ? a.n_dst - d0 : DZ_NB);
    if (wv == 0 && lane <= nd) rps[lane] = a.row_ptr[d0 + lane];
    lds_barrier();
    ntile = (rps[nd] - rps[0] + 31) / 32;
    Tile tA, tB;
    locate(pr, tA);
    load_col(tA);
    locate(4 + pr, tB);
    load_col(tB);
    load_uh(tA, op);
    load_attr(tA, op);
    load_m2(tA, op);
    load_m1(tA, op);
    for (int r0 = 0; r0 < ntile; r0 += 8) {
      round(r0, tA, tB);
      if (r0 + 4 < ntile) round(r0 + 4, tB, tA);
    }
    lds_barrier();   // the block's row pointers are read until every wave is done
  }
  // ---- partial sums of this workgroup (stored positions mapped back to k, j)
  float* o2 = g.p_w2 + (size_t)blockIdx.x * (H2 * H1 + H2);
  if (active) {
    const int j = kperm<__bf16>(jt * 32 + l32);
#pragma unroll
    for (int m = 0; m < G::TPW; ++m) {
      const int kt = kt_of(m);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int k = kperm<__bf16>(kt * 32 + 8 * (i / 4) + 4 * hh + (i % 4));
        o2[(size_t)k * H1 + j] = acc2[m][i];
      }
    }
  }
  {
    const float bs = db2 + __shfl_xor(db2, 32, 64);
    if (bm >= 0 && hh == 0) o2[H2 * H1 + kperm<__bf16>(kt_of(bm) * 32 + l32)] = bs;
  }
  if (wv < JT) {
    float* o1 = g.p_w1 + (size_t)blockIdx.x * (H1 * g.de + H1);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float lo = __shfl_down(acc1[i], 8, 64);
      const int jj = kperm<__bf16>(jt * 32 + 8 * (i / 4) + 4 * hh + (i % 4));
      if (l32 < g.de) o1[(size_t)jj * g.de + l32] = acc1[i] + lo;
      if (l32 == 16) o1[(size_t)H1 * g.de + jj] = acc1[i];
    }
  }
}

struct UArgs {
  int64_t n_rows;
  const unsigned char* G;    // [n_rows][DL] layer dtype (g_i)
  const unsigned char* W;    // [h2*DL][DL] layer dtype: W[k*DL + p][q] = W3[p*DL+q][k]
  unsigned char* U;          // [n_rows][h2*DL] layer dtype, each row in MFMA fragment order
};

// U[i][c] = sum_q W[c][q] g_i[q] for c = k*DL + p, as tiles C[c][i] (A = W
// rows, B = the g rows, lane = destination).  A workgroup owns CB
// consecutive columns (one to four 32-column tiles per wave, whose W rows stay
// in registers for the whole launch) and a range of destinations, taken 32
// at a time: the products land in an LDS block [32 destinations][CB columns]
// (two buffers, one barrier per step) that is stored by whole row pieces
// (512 bytes or 1 KB) with streaming stores.
template <typename T, int DL, int H2>
struct UShape {
  // columns per workgroup: row pieces of 1 KB where U rows are long enough, else 512 bytes
  static constexpr int ESZ = sizeof(T), CB = (H2 * DL >= 8192 ? 1024 : 512) / ESZ;
  static constexpr int TPW = CB / 128;                     // column tiles per wave
  static constexpr int TROW = CB * ESZ + 16;               // LDS row pitch (bytes)
  static constexpr int BUF = 32 * TROW;
};

template <typename T, int DL, int H2>
__global__ __launch_bounds__(256) void k_u_gemm(UArgs a, int64_t rows_per_wg) {
  using M = MT<T>;
  using frag = typename M::frag;
  using US = UShape<T, DL, H2>;
  constexpr int KS = M::KS, EPL = M::EPL, ESZ = sizeof(T), SKD = DL / KS, NC = H2 * DL, TROW = US::TROW;
  constexpr int CB = US::CB, CH = CB * ESZ / 16;          // columns, 16-byte units of an LDS row
  extern __shared__ __align__(16) unsigned char sqm[];
  unsigned char (*sq)[US::BUF] = reinterpret_cast<unsigned char (*)[US::BUF]>(sqm);
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  const int64_t cb0 = (int64_t)blockIdx.x * CB;
  const int64_t i_begin = (int64_t)blockIdx.y * rows_per_wg;
  const int64_t i_end = i_begin + rows_per_wg < a.n_rows ? i_begin + rows_per_wg : a.n_rows;
  frag A[US::TPW][SKD];
#pragma unroll
  for (int m = 0; m < US::TPW; ++m)
#pragma unroll
    for (int s = 0; s < SKD; ++s)
      A[m][s] = ld_frag<T>(a.W + ((size_t)(cb0 + (wv * US::TPW + m) * 32 + l32) * DL + s * KS + hh * EPL) * ESZ);
  // the g rows of a step are loaded one step ahead, ahead of the previous
  // step's stores: loads and stores retire in order, so a load issued after
  // the stores would wait for them too
  frag B[SKD];
  {
    const int64_t row = i_begin + l32 < i_end ? i_begin + l32 : i_end - 1;
#pragma unroll
    for (int s = 0; s < SKD; ++s) B[s] = ld_frag<T>(a.G + ((size_t)row * DL + s * KS + hh * EPL) * ESZ);
  }
  int buf = 0;
  for (int64_t i0 = i_begin; i0 < i_end; i0 += 32, buf ^= 1) {
    unsigned char* t = sq[buf];
#pragma unroll
    for (int m = 0; m < US::TPW; ++m) {
      f32x16 C = f32x16{};
#pragma unroll
      for (int s = 0; s < SKD; ++s) C = M::mma(A[m][s], B[s], C);
      // LDS row = destination (lane), columns 32 (wave tile) + 8(r/4) + 4hh + r%4
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        unsigned char* o = t + l32 * TROW + (32 * (wv * US::TPW + m) + 8 * g + 4 * hh) * ESZ;
        if constexpr (ESZ == 2) {
          const bf16x2 lo = __builtin_convertvector((f32x2){C[4 * g], C[4 * g + 1]}, bf16x2);
          const bf16x2 hi = __builtin_convertvector((f32x2){C[4 * g + 2], C[4 * g + 3]}, bf16x2);
          *reinterpret_cast<uint2*>(o) = make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
        } else {
          *reinterpret_cast<f32x4*>(o) = f32x4{C[4 * g], C[4 * g + 1], C[4 * g + 2], C[4 * g + 3]};
        }
      }
    }
    __syncthreads();   // the block is complete; the other buffer's stores are done
    if (i0 + 32 < i_end) {
      const int64_t row = i0 + 32 + l32 < i_end ? i0 + 32 + l32 : i_end - 1;
#pragma unroll
      for (int s = 0; s < SKD; ++s) B[s] = ld_frag<T>(a.G + ((size_t)row * DL + s * KS + hh * EPL) * ESZ);
    }
    // Each wave-wide store covers whole cache lines of one row piece; U is
    // far larger than the caches and is next read by another kernel, so the
    // stores carry the non-temporal (streaming) hint.
#pragma unroll
    for (int it = 0; it < 32 * CH / 256; ++it) {
      const int id = it * 256 + tid, r = id / CH, ch = id % CH;
      const f32x4 v = *reinterpret_cast<const f32x4*>(t + r * TROW + ch * 16);
      if (i0 + r < i_end)
        __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(a.U + ((size_t)(i0 + r) * NC + cb0) * ESZ + ch * 16));
    }
  }
}

// Launch shape of k_u_gemm: column blocks, destinations split into groups of
// whole 32-row steps so that there are about four workgroups per CU.
template <typename T, int DL, int H2>
dsmp_status launch_u_gemm(dsmp_handle* h, const UArgs& ua) {
  if (ua.n_rows == 0) return DSMP_OK;
  constexpr int NC = H2 * DL, CB = UShape<T, DL, H2>::CB;
  static_assert(NC % CB == 0, "U columns are whole column blocks");
  const int64_t ncb = NC / CB;
  int64_t groups = ((int64_t)h->n_cu * 4 + ncb - 1) / ncb;
  const int64_t steps = (ua.n_rows + 31) / 32;
  if (groups > steps) groups = steps;
  const int64_t rows_per_wg = ((steps + groups - 1) / groups) * 32;
  groups = (ua.n_rows + rows_per_wg - 1) / rows_per_wg;
  constexpr int lds = 2 * UShape<T, DL, H2>::BUF;
  DSMP_HIP(h, hipFuncSetAttribute(reinterpret_cast<const void*>(k_u_gemm<T, DL, H2>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, lds));
  hipLaunchKernelGGL((k_u_gemm<T, DL, H2>), dim3((unsigned)ncb, (unsigned)groups), dim3(256), lds, h->stream, ua,
                     rows_per_wg);
  DSMP_LAUNCHED(h, "U GEMM");
  return DSMP_OK;
}

// Transposed staging of a chunk of ECH edge rows of a [E][W] array (layer
// dtype, permuted register order) into LDS as [W][ECH] (rows still in the
// permuted order), four edges per thread: 8-byte (bf16) or 16-byte (fp32)
// LDS writes, zero rows past e_end.  fetch() loads a chunk into registers
// (issued before the current chunk's products), store() writes it to LDS
// with row pitch ROWB bytes after the barrier.
template <typename T, int W, int ECH>
struct TStage {
  static constexpr int ESZ = sizeof(T), KPU = 16 / ESZ, EQ = ECH / 4, NU = EQ * (W / KPU), UPT = (NU + 255) / 256;
  uint4 v[UPT][4];
  __device__ __forceinline__ void fetch(const unsigned char* __restrict__ src, int64_t eb, int64_t e_end) {
#pragma unroll
    for (int x = 0; x < UPT; ++x) {
      const int u = (int)threadIdx.x + x * 256, eq = u % EQ, kg = u / EQ;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t e = eb + 4 * eq + i;
        v[x][i] = (u < NU && e < e_end) ? *reinterpret_cast<const uint4*>(src + ((size_t)e * W) * ESZ + kg * 16)
                                       : make_uint4(0, 0, 0, 0);
      }
    }
  }
  template <int ROWB>
  __device__ __forceinline__ void store(unsigned char* __restrict__ dstl) const {
#pragma unroll
    for (int x = 0; x < UPT; ++x) {
      const int u = (int)threadIdx.x + x * 256, eq = u % EQ, kg = u / EQ;
      if (u >= NU) continue;
      const uint32_t* d0 = reinterpret_cast<const uint32_t*>(&v[x][0]);
      const uint32_t* d1 = reinterpret_cast<const uint32_t*>(&v[x][1]);
      const uint32_t* d2 = reinterpret_cast<const uint32_t*>(&v[x][2]);
      const uint32_t* d3 = reinterpret_cast<const uint32_t*>(&v[x][3]);
      if constexpr (ESZ == 2) {
#pragma unroll
        for (int w = 0; w < 8; ++w) {
          const int sh = (w & 1) * 16, dw = w >> 1;
          const uint32_t lo = ((d0[dw] >> sh) & 0xFFFFu) | (((d1[dw] >> sh) & 0xFFFFu) << 16);
          const uint32_t hi = ((d2[dw] >> sh) & 0xFFFFu) | (((d3[dw] >> sh) & 0xFFFFu) << 16);
          *reinterpret_cast<uint2*>(dstl + (kg * 8 + w) * ROWB + 4 * eq * ESZ) = make_uint2(lo, hi);
        }
      } else {
#pragma unroll
        for (int w = 0; w < 4; ++w)
          *reinterpret_cast<uint4*>(dstl + (kg * 4 + w) * ROWB + 4 * eq * ESZ) = make_uint4(d0[w], d1[w], d2[w], d3[w]);
      }
    }
  }
};

// ------------------------------------------------------------ dW3 (split over edges)

struct W3Args {
  int64_t E;
  int64_t per_chunk;   // edges per chunk (multiple of 64)
  int nchunk;
  const int32_t* col;
  const int32_t* dst;
  const unsigned char* h_in;
  const float* gF;
  const unsigned char* zE;
  float* part;         // [nchunk][d*d*h2]
};

// Wave tile of the dW3 product: PW values of p x QTW q-tiles x KTW k-tiles.
// Small q/k extents give each wave two p's over one q-tile, so one g
// fragment read from LDS feeds two formed operands.
template <typename T, int DL, int H2>
struct W3Shape {
  static constexpr int KS = MT<T>::KS, EPL = MT<T>::EPL, ESZ = sizeof(T);
  static constexpr int QT = DL / 32, KT = H2 / 32;
  static constexpr int KTW = KT < 4 ? KT : 4;
  static constexpr bool PAIR = QT * (KT / KTW) <= 2;
  static constexpr int QTW = PAIR ? 1 : 2, PW = PAIR ? 2 : 1;
  static constexpr int WPG = (QT / QTW) * (KT / KTW);   // waves per group of PW p's
  static constexpr int PB = (4 / WPG) * PW;             // p's per workgroup
  static constexpr int ECH = 64;
  static constexpr int ZROW = (ECH + 16 / ESZ) * ESZ;   // bytes per row of the z chunk
  static constexpr int FROW = ECH + 4;                   // floats per row of g / h chunks
  static constexpr int LDS = H2 * ZROW + DL * FROW * 4 + PB * FROW * 4;
  // staging units per thread (rounded up)
  static constexpr int ZU = ((ECH / 4) * (H2 * ESZ / 16) + 255) / 256;
  static constexpr int GU = ((ECH / 4) * (DL / 4) + 255) / 256;
  static constexpr int HU = (ECH * PB + 255) / 256;
  static_assert(WPG * (PB / PW) == 4, "four waves per workgroup");
};

template <typename T, int DL, int H2>
__global__ __launch_bounds__(256, (DL <= 64 && H2 * sizeof(T) <= 256) ? 2 : 1) void k_bwd_dW3(W3Args a) {
  using S = W3Shape<T, DL, H2>;
  using M = MT<T>;
  using frag = typename M::frag;
  constexpr int KS = S::KS, EPL = S::EPL, ESZ = S::ESZ, ECH = S::ECH, EQ = ECH / 4;
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* zl = smem;
  float* gl = reinterpret_cast<float*>(smem + H2 * S::ZROW);
  float* hl = gl + DL * S::FROW;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  // workgroups of one edge chunk sit on one XCD (ids congruent mod 8)
  constexpr int NPB = DL / S::PB;
  const int wg = blockIdx.x, xcd = wg & 7, slot = wg >> 3;
  const int chunk = (slot / NPB) * 8 + xcd, pb = slot % NPB;
  const int p0 = pb * S::PB;
  const int grp = wv / S::WPG, sub = wv % S::WPG;
  const int pl0 = grp * S::PW;                                   // first local p of this wave
  const int qt0 = (sub % (S::QT / S::QTW)) * S::QTW, kt0 = (sub / (S::QT / S::QTW)) * S::KTW;
  const T* hin = reinterpret_cast<const T*>(a.h_in);
  const int64_t e_begin = (int64_t)chunk * a.per_chunk;
  int64_t e_end = e_begin + a.per_chunk;
  if (e_end > a.E) e_end = a.E;

  f32x16 acc[S::PW][S::KTW][S::QTW];
#pragma unroll
  for (int pp = 0; pp < S::PW; ++pp)
#pragma unroll
    for (int kk = 0; kk < S::KTW; ++kk)
#pragma unroll
      for (int qq = 0; qq < S::QTW; ++qq) acc[pp][kk][qq] = f32x16{};

  // next chunk held in registers while the current one is multiplied
  uint4 zr[S::ZU][4];
  f32x4 gr[S::GU][4];
  float hr[S::HU];
  auto fetch = [&](int64_t eb) {
#pragma unroll
    for (int x = 0; x < S::ZU; ++x) {
      const int u = tid + x * 256, eq = u % EQ, kg = u / EQ;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t e = eb + 4 * eq + i;
        zr[x][i] = (u < EQ * (H2 * ESZ / 16) && e < e_end)
                       ? *reinterpret_cast<const uint4*>(a.zE + (size_t)e * H2 * ESZ + kg * 16)
                       : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int x = 0; x < S::GU; ++x) {
      const int u = tid + x * 256, eq = u % EQ, q4 = u / EQ;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t e = eb + 4 * eq + i;
        gr[x][i] = (u < EQ * (DL / 4) && e < e_end)
                       ? *reinterpret_cast<const f32x4*>(a.gF + (size_t)a.dst[e] * DL + q4 * 4)
                       : f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
#pragma unroll
    for (int x = 0; x < S::HU; ++x) {
      const int u = tid + x * 256, el = u / S::PB, pp = u % S::PB;
      const int64_t e = eb + el;
      hr[x] = (u < ECH * S::PB && e < e_end) ? to_f(hin[(size_t)a.col[e] * DL + p0 + pp]) : 0.0f;
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int x = 0; x < S::ZU; ++x) {
      const int u = tid + x * 256, eq = u % EQ, kg = u / EQ;
      if (u >= EQ * (H2 * ESZ / 16)) continue;
      const uint32_t* d0 = reinterpret_cast<const uint32_t*>(&zr[x][0]);
      const uint32_t* d1 = reinterpret_cast<const uint32_t*>(&zr[x][1]);
      const uint32_t* d2 = reinterpret_cast<const uint32_t*>(&zr[x][2]);
      const uint32_t* d3 = reinterpret_cast<const uint32_t*>(&zr[x][3]);
      if constexpr (ESZ == 2) {
#pragma unroll
        for (int w = 0; w < 8; ++w) {
          const int sh = (w & 1) * 16, dw = w >> 1;
          const uint32_t lo = ((d0[dw] >> sh) & 0xFFFFu) | (((d1[dw] >> sh) & 0xFFFFu) << 16);
          const uint32_t hi = ((d2[dw] >> sh) & 0xFFFFu) | (((d3[dw] >> sh) & 0xFFFFu) << 16);
          *reinterpret_cast<uint2*>(zl + (kg * 8 + w) * S::ZROW + 4 * eq * ESZ) = make_uint2(lo, hi);
        }
      } else {
#pragma unroll
        for (int w = 0; w < 4; ++w)
          *reinterpret_cast<uint4*>(zl + (kg * 4 + w) * S::ZROW + 4 * eq * ESZ) = make_uint4(d0[w], d1[w], d2[w], d3[w]);
      }
    }
#pragma unroll
    for (int x = 0; x < S::GU; ++x) {
      const int u = tid + x * 256, eq = u % EQ, q4 = u / EQ;
      if (u >= EQ * (DL / 4)) continue;
#pragma unroll
      for (int w = 0; w < 4; ++w)
        *reinterpret_cast<f32x4*>(gl + (q4 * 4 + w) * S::FROW + 4 * eq) =
            f32x4{gr[x][0][w], gr[x][1][w], gr[x][2][w], gr[x][3][w]};
    }
#pragma unroll
    for (int x = 0; x < S::HU; ++x) {
      const int u = tid + x * 256, el = u / S::PB, pp = u % S::PB;
      if (u < ECH * S::PB) hl[pp * S::FROW + el] = hr[x];
    }
  };

  if (e_begin < e_end) fetch(e_begin);
  for (int64_t eb = e_begin; eb < e_end; eb += ECH) {
    __syncthreads();   // the previous chunk's products are done with LDS
    store();
    __syncthreads();
    if (eb + ECH < e_end) fetch(eb + ECH);
#pragma unroll 2
    for (int ks = 0; ks < ECH / KS; ++ks) {
      const int ec = ks * KS + hh * EPL;
      frag A[S::KTW];
#pragma unroll
      for (int kk = 0; kk < S::KTW; ++kk) A[kk] = ld_frag<T>(zl + ((kt0 + kk) * 32 + l32) * S::ZROW + ec * ESZ);
#pragma unroll
      for (int qq = 0; qq < S::QTW; ++qq) {
        const float* gp = gl + ((qt0 + qq) * 32 + l32) * S::FROW + ec;
        float gv[EPL];
#pragma unroll
        for (int u = 0; u < EPL; ++u) gv[u] = gp[u];
#pragma unroll
        for (int pp = 0; pp < S::PW; ++pp) {
          const float* hp = hl + (pl0 + pp) * S::FROW + ec;
          float bv[EPL];
#pragma unroll
          for (int u = 0; u < EPL; ++u) bv[u] = hp[u] * gv[u];
          const frag B = pack_frag<T>(bv);
#pragma unroll
          for (int kk = 0; kk < S::KTW; ++kk) acc[pp][kk][qq] = M::mma(A[kk], B, acc[pp][kk][qq]);
        }
      }
    }
  }
  // tile (rows: stored-order k positions, cols q) -> part[chunk][(p*d + q)*h2 + k]
  float* out = a.part + (size_t)chunk * DL * DL * H2;
#pragma unroll
  for (int pp = 0; pp < S::PW; ++pp) {
    const int p = p0 + pl0 + pp;
#pragma unroll
    for (int qq = 0; qq < S::QTW; ++qq) {
      const int q = (qt0 + qq) * 32 + l32;
      float* o = out + ((size_t)p * DL + q) * H2;
#pragma unroll
      for (int kk = 0; kk < S::KTW; ++kk)
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4) {
          const int r = (kt0 + kk) * 32 + 8 * a4 + 4 * hh;
          if constexpr (EPL == 8) {
            *reinterpret_cast<f32x4*>(o + kperm<T>(r)) = f32x4{acc[pp][kk][qq][4 * a4], acc[pp][kk][qq][4 * a4 + 1],
                                                               acc[pp][kk][qq][4 * a4 + 2], acc[pp][kk][qq][4 * a4 + 3]};
          } else {
#pragma unroll
            for (int b = 0; b < 4; ++b) o[kperm<T>(r + b)] = acc[pp][kk][qq][4 * a4 + b];
          }
        }
    }
  }
}

// ------------------------------------------------------------ dW2 / db2 (split over edges)

struct W2Args {
  int64_t E;
  int64_t per_chunk;
  int nsplit;
  const unsigned char* da2E;   // [E][h2] permuted
  const unsigned char* z1E;    // [E][h1] permuted, or null: recomputed from xE (k_bwd_dW2_rz)
  float* part;                 // [nchunk][h2*h1 + h2]
  const unsigned char* xE;     // [E][32 bytes] bf16 high parts 0..7, low parts 8..15 (k_bwd_dW2_rz)
  const unsigned char* w1l;    // packed W1, fp32 [2][h1/2][8] (k_bwd_dW2_rz)
  const unsigned char* b1l;    // packed b1, fp32 [2][h1/2] (k_bwd_dW2_rz)
};

template <typename T, int H1, int H2>
struct W2Shape {
  static constexpr int KS = MT<T>::KS, EPL = MT<T>::EPL, ESZ = sizeof(T);
  static constexpr int KT = H2 / 32, JT = H1 / 32;
  static constexpr int NSPLIT = KT * JT > 32 ? KT * JT / 32 : 1;
  static constexpr int JT_WG = JT / NSPLIT;                 // j tiles per workgroup
  static constexpr int KT_W = KT >= 4 ? KT / 4 : 1;         // k tiles per wave
  static constexpr int JGRP = KT >= 4 ? 1 : 4 / KT;         // waves sharing one k tile
  static constexpr int JT_W = JT_WG / JGRP;                 // j tiles per wave
  static constexpr int ECH = 64;
  static constexpr int ROW = (ECH + 16 / ESZ) * ESZ;
  static constexpr int LDS = (H2 + H1) * ROW;
};

template <typename T, int H1, int H2>
__global__ __launch_bounds__(256, 2) void k_bwd_dW2(W2Args a) {
  using S = W2Shape<T, H1, H2>;
  using M = MT<T>;
  using frag = typename M::frag;
  constexpr int KS = S::KS, EPL = S::EPL, ESZ = S::ESZ, ECH = S::ECH;
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* dl = smem;                 // da2 [k][e]
  unsigned char* zl = smem + H2 * S::ROW;   // z1 [j][e]
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  const int split = blockIdx.x % S::NSPLIT, chunk = blockIdx.x / S::NSPLIT;
  const int kt0 = (wv / S::JGRP) * S::KT_W;
  const int jt0 = split * S::JT_WG + (wv % S::JGRP) * S::JT_W;
  const int64_t e_begin = (int64_t)chunk * a.per_chunk;
  int64_t e_end = e_begin + a.per_chunk;
  if (e_end > a.E) e_end = a.E;
  f32x16 acc[S::KT_W][S::JT_W];
#pragma unroll
  for (int kk = 0; kk < S::KT_W; ++kk)
#pragma unroll
    for (int jj = 0; jj < S::JT_W; ++jj) acc[kk][jj] = f32x16{};
  float bsum = 0.0f;
  TStage<T, H2, ECH> sa;
  TStage<T, H1, ECH> sz;
  sa.fetch(a.da2E, e_begin, e_end);
  sz.fetch(a.z1E, e_begin, e_end);
  for (int64_t eb = e_begin; eb < e_end; eb += ECH) {
    __syncthreads();
    sa.template store<S::ROW>(dl);
    sz.template store<S::ROW>(zl);
    if (eb + ECH < e_end) {   // next chunk in flight while this one is multiplied
      sa.fetch(a.da2E, eb + ECH, e_end);
      sz.fetch(a.z1E, eb + ECH, e_end);
    }
    __syncthreads();
    if (split == 0 && tid < H2)
      for (int el = 0; el < ECH; ++el) bsum += to_f(*reinterpret_cast<const T*>(dl + tid * S::ROW + el * ESZ));
#pragma unroll 2
    for (int ks = 0; ks < ECH / KS; ++ks) {
      const int ec = ks * KS + hh * EPL;
      frag A[S::KT_W];
#pragma unroll
      for (int kk = 0; kk < S::KT_W; ++kk) A[kk] = ld_frag<T>(dl + ((kt0 + kk) * 32 + l32) * S::ROW + ec * ESZ);
#pragma unroll
      for (int jj = 0; jj < S::JT_W; ++jj) {
        const frag B = ld_frag<T>(zl + ((jt0 + jj) * 32 + l32) * S::ROW + ec * ESZ);
#pragma unroll
        for (int kk = 0; kk < S::KT_W; ++kk) acc[kk][jj] = M::mma(A[kk], B, acc[kk][jj]);
      }
    }
  }
  float* out = a.part + (size_t)chunk * (H2 * H1 + H2);
  // tile rows and columns are stored-order positions; map them back to (k, j)
#pragma unroll
  for (int jj = 0; jj < S::JT_W; ++jj) {
    const int j = kperm<T>((jt0 + jj) * 32 + l32);
#pragma unroll
    for (int kk = 0; kk < S::KT_W; ++kk)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int k = kperm<T>((kt0 + kk) * 32 + 8 * (i / 4) + 4 * hh + (i % 4));
        out[(size_t)k * H1 + j] = acc[kk][jj][i];
      }
  }
  if (split == 0 && tid < H2) out[H2 * H1 + kperm<T>(tid)] = bsum;
}

// bf16: chunks of 64 edge rows of da2 and z1 are copied to LDS as they are
// (whole cache lines, the next chunk in flight while this one is multiplied)
// and the fragments, whose contraction index is the edge, come from
// transposing LDS reads.  Rows past the range re-read its last row and are
// zeroed in the A fragment.
template <int H1, int H2>
struct W2TrShape {
  static constexpr int ECH = 64;
  using DS = RowStage<ECH, H2 * 2, tr_pad_units(H2 * 2)>;
  using ZS = RowStage<ECH, H1 * 2, tr_pad_units(H1 * 2)>;
  static constexpr int DB = ECH * DS::PITCH, BUF = DB + ECH * ZS::PITCH, LDS = 2 * BUF;
};

// W8: eight waves per workgroup cover all (k, j) tiles of a 256 x 256 dW2
// (two k tiles by four j tiles each), so each chunk of edges is read once
// instead of once per half of the j tiles.
template <int H1, int H2, bool W8 = false>
struct W2TrTiles {
  using S = W2Shape<__bf16, H1, H2>;
  static constexpr int NW = W8 ? 8 : 4, NSPLIT = W8 ? 1 : S::NSPLIT;
  static constexpr int KT_W = W8 ? 2 : S::KT_W, JT_W = W8 ? 4 : S::JT_W;
  static_assert(!W8 || (S::KT == 8 && S::JT == 8), "eight waves: h1 = h2 = 256");
};

template <int H1, int H2, bool W8 = false>
__global__ __launch_bounds__(W8 ? 512 : 256, W8 ? 1 : 2) void k_bwd_dW2_tr(W2Args a) {
  using S0 = W2Shape<__bf16, H1, H2>;
  using S = W2TrTiles<H1, H2, W8>;
  using TS = W2TrShape<H1, H2>;
  using M = MT<__bf16>;
  constexpr int ECH = TS::ECH;
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  const int split = blockIdx.x % S::NSPLIT, chunk = blockIdx.x / S::NSPLIT;
  const int kt0 = W8 ? (wv / 2) * 2 : (wv / S0::JGRP) * S0::KT_W;
  const int jt0 = W8 ? (wv % 2) * 4 : split * S0::JT_WG + (wv % S0::JGRP) * S0::JT_W;
  const int64_t e_begin = (int64_t)chunk * a.per_chunk;
  int64_t e_end = e_begin + a.per_chunk;
  if (e_end > a.E) e_end = a.E;
  f32x16 acc[S::KT_W][S::JT_W];
#pragma unroll
  for (int kk = 0; kk < S::KT_W; ++kk)
#pragma unroll
    for (int jj = 0; jj < S::JT_W; ++jj) acc[kk][jj] = f32x16{};
  float bsum = 0.0f;
  if (e_begin < e_end) {   // uniform over the workgroup
    const int nch = (int)((e_end - e_begin + ECH - 1) / ECH);
    typename TS::DS sd;
    typename TS::ZS sz;
    auto issue = [&](int c, unsigned char* buf) {
      if (tid >= 256) return;   // the row stages are laid out for 256 threads
      const int64_t e0 = e_begin + (int64_t)c * ECH;
      const int nv = (int)(e_end - e0 < ECH ? e_end - e0 : ECH);
      sd.init(H2 * 2, nv);
      sz.init(H1 * 2, nv);
      sd.issue(a.da2E + (size_t)e0 * H2 * 2, buf);
      sz.issue(a.z1E + (size_t)e0 * H1 * 2, buf + TS::DB);
    };
    issue(0, smem);
    stage_wait();
    __syncthreads();
    for (int c = 0; c < nch; ++c) {
      const unsigned char* cur = smem + (c & 1) * TS::BUF;
      if (c + 1 < nch) issue(c + 1, smem + ((c + 1) & 1) * TS::BUF);
      const int64_t e0 = e_begin + (int64_t)c * ECH;
      const int cnt = (int)(e_end - e0 < ECH ? e_end - e0 : ECH);
      if (split == 0 && tid < H2)
        for (int e = 0; e < cnt; ++e) bsum += (float)*reinterpret_cast<const __bf16*>(cur + e * TS::DS::PITCH + tid * 2);
      for (int ks = 0; ks < (cnt + 15) / 16; ++ks) {
        bf16x8 A[S::KT_W];
#pragma unroll
        for (int kk = 0; kk < S::KT_W; ++kk) {
          A[kk] = lds_frag_rows(cur, TS::DS::PITCH, ks * 16, (kt0 + kk) * 32);
          if (ks * 16 + 16 > cnt) {
#pragma unroll
            for (int t = 0; t < 8; ++t)
              if (ks * 16 + 8 * hh + t >= cnt) A[kk][t] = (__bf16)0.0f;
          }
        }
#pragma unroll
        for (int jj = 0; jj < S::JT_W; ++jj) {
          const bf16x8 B = lds_frag_rows(cur + TS::DB, TS::ZS::PITCH, ks * 16, (jt0 + jj) * 32);
#pragma unroll
          for (int kk = 0; kk < S::KT_W; ++kk) acc[kk][jj] = M::mma(A[kk], B, acc[kk][jj]);
        }
      }
      stage_wait();
      __syncthreads();
    }
  }
  float* out = a.part + (size_t)chunk * (H2 * H1 + H2);
  // tile rows and columns are stored-order positions; map them back to (k, j)
#pragma unroll
  for (int jj = 0; jj < S::JT_W; ++jj) {
    const int j = kperm<__bf16>((jt0 + jj) * 32 + l32);
#pragma unroll
    for (int kk = 0; kk < S::KT_W; ++kk)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int k = kperm<__bf16>((kt0 + kk) * 32 + 8 * (i / 4) + 4 * hh + (i % 4));
        out[(size_t)k * H1 + j] = acc[kk][jj][i];
      }
  }
  if (split == 0 && tid < H2) out[H2 * H1 + kperm<__bf16>(tid)] = bsum;
}

// dW2 and db2 where the forward kept no z1 rows (d = 128, h1 = h2 = 256):
// z1 = ReLU(W1 x + b1) of each chunk of edges is recomputed on the matrix
// cores from the saved bf16 high and low parts of x, as the fused
// edge-gradient pass does (W1h xh + W1h xl + W1l xh + b1h + b1l with fp32
// accumulation, within about 2^-16 of the forward's fp32 chain), rounded to
// bf16 into the chunk's z1 rows in LDS; the dW2 products, the waves' tiles
// and the outputs are those of k_bwd_dW2_tr with eight waves.  Wave w forms
// the z1 row blocks 2 (w % 4), 2 (w % 4) + 1 of edge block w / 4 of the chunk.
// Two statically distinct chunk buffers alternate in code; the next chunk's
// attribute rows are loaded ahead of its da2 copy.
template <int H1, int H2>
__global__ __launch_bounds__(512, 1) void k_bwd_dW2_rz(W2Args a) {
  using S = W2TrTiles<H1, H2, true>;
  using TS = W2TrShape<H1, H2>;
  using M = MT<__bf16>;
  constexpr int ECH = TS::ECH;
  static_assert(ECH == 64 && H1 == 256, "two 32-edge blocks per chunk, eight 32-row blocks of z1 per block");
  __shared__ __align__(16) unsigned char XA[TS::BUF], XB[TS::BUF];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  const int kt0 = (wv / 2) * 2, jt0 = (wv % 2) * 4, sb = wv / 4;
  const int64_t e_begin = (int64_t)blockIdx.x * a.per_chunk;
  int64_t e_end = e_begin + a.per_chunk;
  if (e_end > a.E) e_end = a.E;
  if (e_begin >= e_end) return;   // uniform over the workgroup (the launch has no empty chunk)
  // A operands of the z1 products: row R of block zb holds the layer-1
  // weights of stored position (2 zb + i/8)*16 + hr*8 + i%8, R = 8(i/4) +
  // 4 hr + i%4; K slots 0..7 W1h, 8..15 W1h, 16..23 W1l, 24 b1h, 25 b1l
  bf16x8 wa[2], wb[2];
  {
    const float* w1 = reinterpret_cast<const float*>(a.w1l);
    const float* b1 = reinterpret_cast<const float*>(a.b1l);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int zb = 2 * (wv % 4) + q;
      const int R = l32, i = 4 * (R / 8) + R % 4, hr = (R % 8) / 4;
      const int pos = (2 * zb + i / 8) * 16 + hr * 8 + i % 8;
      const int hn = ((pos % 16) / 8) * (H1 / 2) + (pos / 16) * 8 + pos % 8;
      const f32x4 w0 = *reinterpret_cast<const f32x4*>(w1 + hn * 8);
      const f32x4 w4 = *reinterpret_cast<const f32x4*>(w1 + hn * 8 + 4);
      const float wvv[8] = {w0[0], w0[1], w0[2], w0[3], w4[0], w4[1], w4[2], w4[3]};
      const float bb = b1[hn];
      float v0[8], v1[8];
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const float whi = (float)(__bf16)wvv[c];
        v0[c] = whi;                          // slots 0..7 (times xh) and 8..15 (times xl)
        v1[c] = hh ? 0.0f : wvv[c] - whi;     // slots 16..23 (times xh)
      }
      if (hh) {
        const float bhi = (float)(__bf16)bb;
        v1[0] = bhi;
        v1[1] = bb - bhi;
      }
      wa[q] = pack_frag<__bf16>(v0);
      wb[q] = pack_frag<__bf16>(v1);
    }
  }
  f32x16 acc[S::KT_W][S::JT_W];
#pragma unroll
  for (int kk = 0; kk < S::KT_W; ++kk)
#pragma unroll
    for (int jj = 0; jj < S::JT_W; ++jj) acc[kk][jj] = f32x16{};
  float bsum = 0.0f;
  const int nch = (int)((e_end - e_begin + ECH - 1) / ECH);
  typename TS::DS sd;
  auto issue = [&](int c, unsigned char* buf) {
    if (tid >= 256) return;   // the row stage is laid out for 256 threads
    const int64_t e0 = e_begin + (int64_t)c * ECH;
    const int nv = (int)(e_end - e0 < ECH ? e_end - e0 : ECH);
    sd.init(H2 * 2, nv);
    sd.issue(a.da2E + (size_t)e0 * H2 * 2, buf);
  };
  // the lane's attribute half-row of its edge in block sb of chunk c
  // (rows past the end re-read the last edge: their products are never used)
  auto xload = [&](int c) -> uint4 {
    int64_t e = e_begin + (int64_t)c * ECH + 32 * sb + l32;
    if (e > e_end - 1) e = e_end - 1;
    return *reinterpret_cast<const uint4*>(a.xE + (size_t)e * 32 + 16 * hh);
  };
  auto zfill = [&](const uint4& xr, unsigned char* buf) {
    const bf16x8 xb0 = __builtin_bit_cast(bf16x8, xr);   // [xh | xl] by lane half
    float one[8] = {1.0f, 1.0f, 0, 0, 0, 0, 0, 0};
    const bf16x8 xb1 = hh ? pack_frag<__bf16>(one) : xb0;   // [xh | 1 1 0 ...]
    unsigned char* zrow = buf + TS::DB + (32 * sb + l32) * TS::ZS::PITCH;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int zb = 2 * (wv % 4) + q;
      f32x16 Z = f32x16{};
      Z = M::mma(wa[q], xb0, Z);
      Z = M::mma(wb[q], xb1, Z);
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        float zv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) zv[u] = relu_bits(Z[8 * r + u]);
        *reinterpret_cast<bf16x8*>(zrow + ((2 * zb + r) * 16 + hh * 8) * 2) = pack_frag<__bf16>(zv);
      }
    }
  };
  auto products = [&](int c, const unsigned char* cur) {
    const int64_t e0 = e_begin + (int64_t)c * ECH;
    const int cnt = (int)(e_end - e0 < ECH ? e_end - e0 : ECH);
    if (tid < H2)
      for (int e = 0; e < cnt; ++e) bsum += (float)*reinterpret_cast<const __bf16*>(cur + e * TS::DS::PITCH + tid * 2);
    for (int ks = 0; ks < (cnt + 15) / 16; ++ks) {
      bf16x8 A[S::KT_W];
#pragma unroll
      for (int kk = 0; kk < S::KT_W; ++kk) {
        A[kk] = lds_frag_rows(cur, TS::DS::PITCH, ks * 16, (kt0 + kk) * 32);
        if (ks * 16 + 16 > cnt) {
#pragma unroll
          for (int t = 0; t < 8; ++t)
            if (ks * 16 + 8 * hh + t >= cnt) A[kk][t] = (__bf16)0.0f;
        }
      }
#pragma unroll
      for (int jj = 0; jj < S::JT_W; ++jj) {
        const bf16x8 B = lds_frag_rows(cur + TS::DB, TS::ZS::PITCH, ks * 16, (jt0 + jj) * 32);
#pragma unroll
        for (int kk = 0; kk < S::KT_W; ++kk) acc[kk][jj] = M::mma(A[kk], B, acc[kk][jj]);
      }
    }
  };
  // one chunk: its da2 rows copied and z1 rows written (cur); the next
  // chunk's attribute rows, then its da2 copy, go out ahead of the products;
  // its z1 rows are written after them
  auto step = [&](int c, const unsigned char* cur, unsigned char* nxt) {
    uint4 xr = make_uint4(0, 0, 0, 0);
    if (c + 1 < nch) {
      xr = xload(c + 1);
      issue(c + 1, nxt);
    }
    products(c, cur);
    if (c + 1 < nch) zfill(xr, nxt);
    stage_wait();
    __syncthreads();
  };
  {
    const uint4 xr = xload(0);
    issue(0, XA);
    zfill(xr, XA);
    stage_wait();
    __syncthreads();
  }
  for (int c = 0;;) {
    step(c, XA, XB);
    if (++c >= nch) break;
    step(c, XB, XA);
    if (++c >= nch) break;
  }
  float* out = a.part + (size_t)blockIdx.x * (H2 * H1 + H2);
  // tile rows and columns are stored-order positions; map them back to (k, j)
#pragma unroll
  for (int jj = 0; jj < S::JT_W; ++jj) {
    const int j = kperm<__bf16>((jt0 + jj) * 32 + l32);
#pragma unroll
    for (int kk = 0; kk < S::KT_W; ++kk)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int k = kperm<__bf16>((kt0 + kk) * 32 + 8 * (i / 4) + 4 * hh + (i % 4));
        out[(size_t)k * H1 + j] = acc[kk][jj][i];
      }
  }
  if (tid < H2) out[H2 * H1 + kperm<__bf16>(tid)] = bsum;
}

// ------------------------------------------------------------ dW1 / db1 (split over edges)

template <typename T, int H1>
__global__ __launch_bounds__(256) void k_bwd_dW1(int64_t E, int64_t per_chunk, const int32_t* __restrict__ col,
                                                 const int32_t* __restrict__ dst, const float* __restrict__ node_attr,
                                                 int dim, int attr_mode, int de, const T* __restrict__ da1E,
                                                 float* __restrict__ part) {
  constexpr int SUB = 256 / H1, XB = 256;
  __shared__ float xs[XB][9];
  __shared__ float red[SUB][H1][9];
  const int kk = threadIdx.x % H1, sub = threadIdx.x / H1;
  const int64_t e0 = (int64_t)blockIdx.x * per_chunk;
  int64_t e1 = e0 + per_chunk;
  if (e1 > E) e1 = E;
  float acc[9];
#pragma unroll
  for (int c = 0; c < 9; ++c) acc[c] = 0.0f;
  for (int64_t eb = e0; eb < e1; eb += XB) {
    __syncthreads();
    {
      const int64_t e = eb + threadIdx.x;
      float x[8];
      if (e < e1) edge_attr(node_attr, dim, attr_mode, dst[e], col[e], x);
#pragma unroll
      for (int c = 0; c < 8; ++c) xs[threadIdx.x][c] = e < e1 ? x[c] : 0.0f;
      xs[threadIdx.x][8] = e < e1 ? 1.0f : 0.0f;
    }
    __syncthreads();
    const int n = e1 - eb < XB ? (int)(e1 - eb) : XB;
#pragma unroll 4
    for (int u = sub; u < n; u += SUB) {
      const float v = to_f(da1E[(eb + u) * H1 + kk]);
#pragma unroll
      for (int c = 0; c < 9; ++c) acc[c] += v * xs[u][c];
    }
  }
#pragma unroll
  for (int c = 0; c < 9; ++c) red[sub][kk][c] = acc[c];
  __syncthreads();
  if (sub == 0) {
    for (int s = 1; s < SUB; ++s)
#pragma unroll
      for (int c = 0; c < 9; ++c) acc[c] += red[s][kk][c];
    const int j = sizeof(T) == 2 ? kperm<__bf16>(kk) : kperm<float>(kk);
    float* out = part + (size_t)blockIdx.x * (H1 * de + H1);
    for (int c = 0; c < de; ++c) out[j * de + c] = acc[c];
    out[H1 * de + j] = acc[8];
  }
}

// bf16 layers: dW1[j][c] = sum_e da1[e][j] x_e[c] on MFMA.  Chunks of 64 edge
// rows of da1 and of the saved attributes (bf16 high parts in columns 0..7,
// low parts in 8..15) are copied to LDS by whole rows, double-buffered; the
// two column halves added restore the attributes to about 16 bits.  Rows
// past the range re-read its last row and are zeroed in the A fragment.
// db1 sums the da1 rows.
template <int H1>
struct W1TrShape {
  static constexpr int ECH = 64;
  using AS = RowStage<ECH, H1 * 2, tr_pad_units(H1 * 2)>;
  using XS = RowStage<ECH, 32, tr_pad_units(32)>;   // 32 bytes of attributes per row, pitch 64
  static constexpr int AB = ECH * AS::PITCH, BUF = AB + ECH * XS::PITCH, LDS = 2 * BUF;
  static constexpr int JT = H1 / 32, JTW = (JT + 3) / 4;
};

template <int H1>
__global__ __launch_bounds__(256) void k_bwd_dW1_tr(int64_t E, int64_t per_chunk, const unsigned char* __restrict__ da1E,
                                                    const unsigned char* __restrict__ xE, int de,
                                                    float* __restrict__ part) {
  using S = W1TrShape<H1>;
  using M = MT<__bf16>;
  constexpr int ECH = S::ECH;
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  const int64_t e_begin = (int64_t)blockIdx.x * per_chunk;
  int64_t e_end = e_begin + per_chunk;
  if (e_end > E) e_end = E;
  f32x16 acc[S::JTW];
#pragma unroll
  for (int jw = 0; jw < S::JTW; ++jw) acc[jw] = f32x16{};
  float bsum = 0.0f;
  if (e_begin < e_end) {   // uniform over the workgroup
    const int nch = (int)((e_end - e_begin + ECH - 1) / ECH);
    typename S::AS sa;
    typename S::XS sx;
    auto issue = [&](int c, unsigned char* buf) {
      const int64_t e0 = e_begin + (int64_t)c * ECH;
      const int nv = (int)(e_end - e0 < ECH ? e_end - e0 : ECH);
      sa.init(H1 * 2, nv);
      sx.init(32, nv);
      sa.issue(da1E + (size_t)e0 * H1 * 2, buf);
      sx.issue(xE + (size_t)e0 * 32, buf + S::AB);
    };
    issue(0, smem);
    stage_wait();
    __syncthreads();
    for (int c = 0; c < nch; ++c) {
      const unsigned char* cur = smem + (c & 1) * S::BUF;
      if (c + 1 < nch) issue(c + 1, smem + ((c + 1) & 1) * S::BUF);
      const int64_t e0 = e_begin + (int64_t)c * ECH;
      const int cnt = (int)(e_end - e0 < ECH ? e_end - e0 : ECH);
      if (tid < H1)
        for (int e = 0; e < cnt; ++e) bsum += (float)*reinterpret_cast<const __bf16*>(cur + e * S::AS::PITCH + tid * 2);
      for (int ks = 0; ks < (cnt + 15) / 16; ++ks) {
        const bf16x8 B = lds_frag_rows(cur + S::AB, S::XS::PITCH, ks * 16, 0);
#pragma unroll
        for (int jw = 0; jw < S::JTW; ++jw) {
          const int jt = wv + 4 * jw;
          if (jt < S::JT) {
            bf16x8 A = lds_frag_rows(cur, S::AS::PITCH, ks * 16, jt * 32);
            if (ks * 16 + 16 > cnt) {
#pragma unroll
              for (int t = 0; t < 8; ++t)
                if (ks * 16 + 8 * hh + t >= cnt) A[t] = (__bf16)0.0f;
            }
            acc[jw] = M::mma(A, B, acc[jw]);
          }
        }
      }
      stage_wait();
      __syncthreads();
    }
  }
  float* out = part + (size_t)blockIdx.x * (H1 * de + H1);
  // column c of a tile holds the high-part sums, column c + 8 the low-part sums
#pragma unroll
  for (int jw = 0; jw < S::JTW; ++jw) {
    const int jt = wv + 4 * jw;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float lo = __shfl_down(acc[jw][i], 8, 64);
      if (jt < S::JT && l32 < de) {
        const int j = kperm<__bf16>(jt * 32 + 8 * (i / 4) + 4 * hh + (i % 4));
        out[(size_t)j * de + l32] = acc[jw][i] + lo;
      }
    }
  }
  if (tid < H1) out[H1 * de + kperm<__bf16>(tid)] = bsum;
}

// ------------------------------------------------------------ attribute gradient

// Diff-mode edge attributes x_e = v_i - v_j: dL/dx_e = W1^T da1_e.  Sixteen
// lanes per edge, each over H1/16 consecutive stored positions of the edge's
// da1 row; W1 in the packed lane order (stored position kk is lane-order
// entry ((kk % KS) / EPL) * H1/2 + (kk / KS) * EPL + kk % EPL), in LDS.
template <typename T, int H1>
__global__ __launch_bounds__(256) void k_attr_dx(int64_t E, const unsigned char* __restrict__ da1E,
                                                 const float* __restrict__ w1l, float4* __restrict__ dx) {
  constexpr int KS = MT<T>::KS, EPL = MT<T>::EPL, PER = H1 / 16;
  __shared__ float w1s[H1 * 8];
  for (int x = threadIdx.x; x < H1 * 8; x += 256) w1s[x] = w1l[x];
  __syncthreads();
  const int g = threadIdx.x & 15;
  // the 16 lanes of an edge are active together, so the shuffles stay within live lanes
  for (int64_t e = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 4; e < E; e += (int64_t)gridDim.x * 16) {
    const T* row = reinterpret_cast<const T*>(da1E) + e * H1 + g * PER;
    float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int t = 0; t < PER; ++t) {
      const int kk = g * PER + t;
      const int hn = ((kk % KS) / EPL) * (H1 / 2) + (kk / KS) * EPL + kk % EPL;
      const float v = to_f(row[t]);
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[c] = __builtin_fmaf(w1s[hn * 8 + c], v, acc[c]);
    }
#pragma unroll
    for (int o = 8; o >= 1; o >>= 1)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[c] += __shfl_xor(acc[c], o, 16);
    if (g == 0) dx[e] = make_float4(acc[0], acc[1], acc[2], acc[3]);
  }
}

// dattr[n] (+)= sum of dx over the edges into n, minus the sum over the edges
// out of n.  Sixteen lanes per node: lane g takes every 16th edge of each
// list, then a fixed butterfly adds the lanes (a fixed order).
__global__ __launch_bounds__(256) void k_attr_seg(int64_t n_src, int64_t n_dst, int de,
                                                  const int32_t* __restrict__ row_ptr,
                                                  const int32_t* __restrict__ csc_ptr,
                                                  const int32_t* __restrict__ csc_eid, const float4* __restrict__ dx,
                                                  float* __restrict__ dattr, int accumulate) {
  const int64_t n = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 4;
  const int g = threadIdx.x & 15;
  if (n >= n_src) return;   // whole 16-lane groups leave together
  float s[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (n < n_dst)
    for (int32_t e = row_ptr[n] + g; e < row_ptr[n + 1]; e += 16) {
      const float4 v = dx[e];
      s[0] += v.x; s[1] += v.y; s[2] += v.z; s[3] += v.w;
    }
  for (int32_t k = csc_ptr[n] + g; k < csc_ptr[n + 1]; k += 16) {
    const float4 v = dx[csc_eid[k]];
    s[0] -= v.x; s[1] -= v.y; s[2] -= v.z; s[3] -= v.w;
  }
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1)
#pragma unroll
    for (int c = 0; c < 4; ++c) s[c] += __shfl_xor(s[c], o, 16);
  if (g < de) {
    const float v = g == 0 ? s[0] : g == 1 ? s[1] : g == 2 ? s[2] : s[3];
    float* o = dattr + n * de + g;
    *o = accumulate ? *o + v : v;
  }
}

template <typename T, int H1>
dsmp_status launch_attr_dx(dsmp_handle* h, int64_t E, const unsigned char* da1E, const float* w1l, float4* dx) {
  const int64_t grid = std::min<int64_t>(ceil_div(E, 16), (int64_t)h->n_cu * 8);
  hipLaunchKernelGGL((k_attr_dx<T, H1>), dim3((unsigned)grid), dim3(256), 0, h->stream, E, da1E, w1l, dx);
  DSMP_LAUNCHED(h, "edge-attribute gradient");
  return DSMP_OK;
}

// ------------------------------------------------------------ reductions and finals

// Fixed-order reductions out[x] = [out[x] +] sum_c part[c*stride + off + x]
// for several segments in one launch: block b serves the 64 outputs starting
// at (b - first[s]) * 64 of segment s; sixteen thread groups sum the chunks
// c = g, g+16, ... in order and the group sums are added in group order
// (deterministic).
struct RedSeg {
  const float* part;
  float* out;
  int64_t stride, off, n;
  int nchunk;
};
struct RedArgs {
  RedSeg seg[8];
  int64_t first[9];
  int nseg, accumulate;
};

constexpr int RED_GROUPS = 16;

__global__ __launch_bounds__(64 * RED_GROUPS) void k_reduce_multi(RedArgs a) {
  __shared__ float sh[RED_GROUPS][64];
  int sidx = 0;
  while (sidx + 1 < a.nseg && (int64_t)blockIdx.x >= a.first[sidx + 1]) ++sidx;
  const RedSeg& sg = a.seg[sidx];
  const int c0 = threadIdx.x & 63, g = threadIdx.x >> 6;
  const int64_t x = ((int64_t)blockIdx.x - a.first[sidx]) * 64 + c0;
  float sum = 0.0f;
  if (x < sg.n && g < sg.nchunk)
    sum = ordered_sum(sg.part + sg.off + x + (int64_t)g * sg.stride, RED_GROUPS * sg.stride,
                      (sg.nchunk - g + RED_GROUPS - 1) / RED_GROUPS);
  sh[g][c0] = sum;
  __syncthreads();
  if (g == 0 && x < sg.n) {
    float t = sh[0][c0];
#pragma unroll
    for (int u = 1; u < RED_GROUPS; ++u) t += sh[u][c0];
    sg.out[x] = a.accumulate ? sg.out[x] + t : t;
  }
}

__device__ __forceinline__ float segment_sum(const int32_t* __restrict__ ptr, int64_t i, int q, int DL,
                                             const float* __restrict__ direct, const float* __restrict__ part) {
  const int64_t pa = ptr[i], pb = ptr[i + 1];
  if (pb <= pa) return 0.0f;
  const int64_t ta = pa / EDGE_TILE, tb = (pb - 1) / EDGE_TILE;
  if (ta == tb) return direct[i * DL + q];
  float s = part[(ta * 2 + 1) * DL + q];
  for (int64_t t = ta + 1; t < tb; ++t) s += part[(t * 2) * DL + q];
  s += part[(tb * 2) * DL + q];
  return s;
}

// grad_h[j] = [root/residual terms if j is a destination] + sum over the edges leaving j
// (aggregate form: the edge sum is the nsl K-slices of the W3 GEMM over T)
__global__ void k_bwd_dh_final(int64_t n_src, int64_t n_dst, int DL, const int32_t* __restrict__ csc_ptr,
                               const float* __restrict__ direct, const float* __restrict__ part, int nsl,
                               const float* __restrict__ slices, const float* __restrict__ dh_node,
                               float* __restrict__ grad_h) {
  const int64_t total = n_src * DL;
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < total; x += (int64_t)gridDim.x * blockDim.x) {
    const int64_t j = x / DL;
    const int c = (int)(x % DL);
    float s = 0.0f;
    if (nsl > 0) {
      s = ordered_sum(slices + x, total, nsl);
    } else {
      s = segment_sum(csc_ptr, j, c, DL, direct, part);
    }
    if (j < n_dst) s += dh_node[x];
    grad_h[x] = s;
  }
}


// ------------------------------------------------------------ feature gradient from U
// The feature gradient of the aggregate form (bf16) without per-source sums:
// for the edge e = (i <- j),
//   sum_q Theta_e[p][q] g_i[q] = sum_k z~_e[k] U~_i[k][p],
// U~_i[k][p] = sum_q W3~[p*d+q][k] g_i[q] -- the same U_i the dz pass reads,
// plus the bias row k = h2, sum_q b3[p*d+q] g_i[q].  k_dh_u forms these
// per-edge terms m_e[p] for every edge of a destination, U_i staged once in
// LDS (rows in the stored order of z, so the z rows load as they are);
// k_dh_gather then sums them over the edges leaving each source, in edge
// order, and adds the node terms.
struct DhuArgs {
  int64_t n_dst;
  const int32_t* row_ptr;
  const unsigned char* U;     // [n_dst][h2*d] bf16, each row in MFMA fragment order
  const unsigned char* gT;    // [n_dst][d] bf16
  const unsigned char* b3n;   // [d][d] bf16, b3[p*d + q]
  const unsigned char* zE;    // [E][h2] bf16, stored positions
  unsigned char* mE;          // [E][d] bf16 out
};

template <int DL, int H2>
struct DhuShape {
  static constexpr int UB = H2 * DL * 2;   // bytes of one U_i (bf16, MFMA fragment order)
  static constexpr int LDS = 2 * UB;       // two destinations' U_i: one in use, the next one arriving
  static_assert(UB % (256 * 16) == 0, "U_i is whole rounds of 256 16-byte units");
};

// U row R of a 32-row tile holds the neuron of z position swap(R): the dz
// pass's accumulator row 8(i/4) + 4h + i%4 is stored at 16(i/8) + 8h + i%8,
// which exchanges bits 2 and 3 of the row within its tile.
__device__ __forceinline__ int swap_bits23(int r) { return (r & ~12) | ((r >> 2) & 1) << 3 | ((r >> 3) & 1) << 2; }

// Byte offset of U_i[R][p .. p+3] (p a multiple of 4) in the fragment order
// of the U GEMM: fragment (kt, s) = 64 lanes x 8 elements, lane r + 32 h
// holding row 32 kt + r, columns 16 s + 8 h .. + 7.
template <int DL>
__device__ __forceinline__ int u_offset(int R, int p) {
  constexpr int SKD = DL / 16;
  return ((((R >> 5) * SKD + (p >> 4)) * 64 + (R & 31) + 32 * ((p >> 3) & 1)) * 8 + (p & 7)) * 2;
}

// A operand of m_e = U_i^T z~_e: lane (n = l%32, h = l/32) receives
// U_i[R(P)][c0 + n] for P = P0 + 8h + t, t < 8, with R(P) the U row of z
// position P -- two transposing LDS reads whose lanes name their own rows in
// the fragment-order copy of U_i (see lds_frag_rows for the lane pattern).
template <int DL>
__device__ __forceinline__ bf16x8 lds_frag_ut(const unsigned char* X, int P0, int c0) {
  const int l = threadIdx.x & 63, g = l >> 4, j = (l >> 2) & 3, q = l & 3;
  const int Plo = P0 + 8 * (g >> 1) + j, Phi = Plo + 4, p = c0 + 16 * (g & 1) + 4 * q;
  const int Rlo = (Plo & ~31) | swap_bits23(Plo & 31), Rhi = (Phi & ~31) | swap_bits23(Phi & 31);
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(X + u_offset<DL>(Rlo, p)));
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(X + u_offset<DL>(Rhi, p)));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Persistent workgroups walk destinations i = blockIdx.x, + gridDim.x, ...:
// U_i is copied to LDS as it stands (direct global-to-LDS loads).  Each wave
// takes (32-row column tile pt of p, 32-edge tile) items of a destination;
// pt is the same for every item of a wave (4 waves, PT divides 4), so the
// bias fragments of b3 are loaded once.  While destination i is multiplied,
// the next destination's U and the operands of the wave's first item of it
// (its z rows and g) are already on their way, so the loop waits on one
// round of loads per destination.
template <int DL, int H2>
__global__ __launch_bounds__(256) void k_dh_u(DhuArgs a) {
  using S = DhuShape<DL, H2>;
  using M = MT<__bf16>;
  constexpr int SKD = DL / 16, SK2 = H2 / 16, PT = DL / 32, NU = S::UB / 16, EPW = 4 / PT;
  static_assert(4 % PT == 0, "column tiles divide the waves");
  extern __shared__ __align__(16) unsigned char X[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  const int pt = wv % PT, et0 = wv / PT;   // the wave's column tile and first edge tile
  bf16x8 ba[SKD];
#pragma unroll
  for (int sf = 0; sf < SKD; ++sf)
    ba[sf] = ld_frag<__bf16>(a.b3n + ((size_t)(32 * pt + l32) * DL + 16 * sf + 8 * hh) * 2);
  // operands of the wave's first item of destination i: z rows of edge tile et0, and g_i
  auto load_ops = [&](int64_t i, int64_t pa, int64_t pb, bf16x8 (&zb)[SK2], bf16x8 (&gb)[SKD]) {
    const int64_t e = pa + (int64_t)et0 * 32 + l32;
    const bool valid = e < pb;
    const unsigned char* zr = a.zE + (size_t)(valid ? e : 0) * H2 * 2;
#pragma unroll
    for (int s2 = 0; s2 < SK2; ++s2) zb[s2] = valid ? ld_frag<__bf16>(zr + (16 * s2 + 8 * hh) * 2) : bf16x8{};
#pragma unroll
    for (int sf = 0; sf < SKD; ++sf) gb[sf] = ld_frag<__bf16>(a.gT + ((size_t)i * DL + 16 * sf + 8 * hh) * 2);
  };
  auto item = [&](const unsigned char* Xb, int64_t pa, int64_t pb, int et, const bf16x8 (&zb)[SK2],
                  const bf16x8 (&gb)[SKD]) {
    const int64_t e = pa + (int64_t)et * 32 + l32;
    f32x16 acc = f32x16{};
    // bias row: sum_q b3[p*d+q] g_i[q], the same for every edge column
#pragma unroll
    for (int sf = 0; sf < SKD; ++sf) acc = M::mma(ba[sf], gb[sf], acc);
#pragma unroll
    for (int s2 = 0; s2 < SK2; ++s2) acc = M::mma(lds_frag_ut<DL>(Xb, 16 * s2, 32 * pt), zb[s2], acc);
    if (e < pb) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const bf16x2 lo = __builtin_convertvector((f32x2){acc[4 * g], acc[4 * g + 1]}, bf16x2);
        const bf16x2 hi = __builtin_convertvector((f32x2){acc[4 * g + 2], acc[4 * g + 3]}, bf16x2);
        *reinterpret_cast<uint2*>(a.mE + ((size_t)e * DL + 32 * pt + 8 * g + 4 * hh) * 2) =
            make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
      }
    }
  };
  int64_t i = blockIdx.x;
  if (i >= a.n_dst) return;
  int64_t pa = a.row_ptr[i], pb = a.row_ptr[i + 1];
  bf16x8 zb[SK2], gb[SKD];
  lds_copy_async<LDS_COPY_STREAM>(a.U + (size_t)i * S::UB, X, NU);   // U_i: last read, streaming
  load_ops(i, pa, pb, zb, gb);
  static_assert(SK2 + SKD < 64, "wait count");
  for (int buf = 0; i < a.n_dst; i += gridDim.x, buf ^= 1) {
    // the copy of U_i was followed by at least SK2 + SKD loads of this thread
    // (its operands): once no more than those are outstanding the copy is in
    // (the item's stores need not have completed)
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(SK2 + SKD));
    __syncthreads();   // U_i is in X[buf]; every wave is done with X[buf ^ 1]
    const unsigned char* Xb = X + buf * S::UB;
    const int64_t inext = i + gridDim.x;
    int64_t pa2 = 0, pb2 = 0;
    bf16x8 zn[SK2], gn[SKD];
    if (inext < a.n_dst) {
      lds_copy_async<LDS_COPY_STREAM>(a.U + (size_t)inext * S::UB, X + (buf ^ 1) * S::UB, NU);
      pa2 = a.row_ptr[inext];
      pb2 = a.row_ptr[inext + 1];
      load_ops(inext, pa2, pb2, zn, gn);
    }
    const int net = (int)((pb - pa + 31) / 32);
    if (et0 < net) item(Xb, pa, pb, et0, zb, gb);
    for (int et = et0 + EPW; et < net; et += EPW) {   // destinations of more than 4 / PT edge tiles
      bf16x8 zx[SK2];
      const int64_t e = pa + (int64_t)et * 32 + l32;
      const unsigned char* zr = a.zE + (size_t)(e < pb ? e : 0) * H2 * 2;
#pragma unroll
      for (int s2 = 0; s2 < SK2; ++s2) zx[s2] = e < pb ? ld_frag<__bf16>(zr + (16 * s2 + 8 * hh) * 2) : bf16x8{};
      item(Xb, pa, pb, et, zx, gb);
    }
#pragma unroll
    for (int s2 = 0; s2 < SK2; ++s2) zb[s2] = zn[s2];
#pragma unroll
    for (int sf = 0; sf < SKD; ++sf) gb[sf] = gn[sf];
    pa = pa2;
    pb = pb2;
  }
}

// grad_h[j] = sum over the edges leaving j of m_e, plus the root and residual
// terms when j is a destination.  One wave per source: the edge ids come in
// with one load per 64 edges and are passed round by shuffles; lanes take two
// channels each, and at d < 128 the wave's lanes form G = 128 / d groups that
// take every G-th edge, their sums then added in group order (a fixed order).
template <int DL>
__global__ __launch_bounds__(256) void k_dh_gather(int64_t n_src, int64_t n_dst, const int32_t* __restrict__ csc_ptr,
                                                   const int32_t* __restrict__ csc_eid,
                                                   const unsigned char* __restrict__ mE,
                                                   const float* __restrict__ dh_node, float* __restrict__ grad_h) {
  constexpr int HW = DL / 2, G = 64 / HW, UN = 8;
  const int lane = threadIdx.x & 63, cp = lane % HW, grp = lane / HW;
  for (int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); j < n_src; j += (int64_t)gridDim.x * 4) {
    const int t0 = csc_ptr[j], t1 = csc_ptr[j + 1];
    float s0 = 0.0f, s1 = 0.0f;
    for (int base = t0; base < t1; base += 64) {
      const int cnt = t1 - base < 64 ? t1 - base : 64;
      const int my = lane < cnt ? csc_eid[base + lane] : 0;
      for (int k = 0; k < cnt; k += G * UN) {
        bf16x2 m[UN];
#pragma unroll
        for (int u = 0; u < UN; ++u) {
          const int idx = k + u * G + grp;
          const int eid = __shfl(my, idx < 64 ? idx : 0, 64);
          m[u] = idx < cnt ? *reinterpret_cast<const bf16x2*>(mE + ((size_t)eid * DL + 2 * cp) * 2) : bf16x2{};
        }
#pragma unroll
        for (int u = 0; u < UN; ++u) {
          s0 += (float)m[u][0];
          s1 += (float)m[u][1];
        }
      }
    }
    // groups in order: group 0 adds group 1's sums, then group 2's, ...
    const float g0 = s0, g1 = s1;
#pragma unroll
    for (int g = 1; g < G; ++g) {
      const float o0 = __shfl(g0, cp + g * HW, 64), o1 = __shfl(g1, cp + g * HW, 64);
      s0 += o0;
      s1 += o1;
    }
    if (grp == 0) {
      if (j < n_dst) {
        s0 += dh_node[j * DL + 2 * cp];
        s1 += dh_node[j * DL + 2 * cp + 1];
      }
      *reinterpret_cast<f32x2*>(grad_h + j * DL + 2 * cp) = f32x2{s0, s1};
    }
  }
}

// ------------------------------------------------------------ dz and feature-gradient terms in one pass
// The two per-edge products that read U_i, dz_e = U_i h_j and
// m_e = U~_i^T z~_e, in one pass over each destination's edges (bf16 layers
// whose kernel-MLP gradients are not fused, h2 = 256), so that U is read from
// HBM once for both.  U_i and g_i are copied to LDS as they stand (direct
// global-to-LDS loads, double-buffered over destinations).  Of the four
// waves, wave w takes, for every 32-edge tile of the destination, the two
// 32-neuron tiles 2w, 2w + 1 of dz (A = U_i fragments read from LDS as
// stored, B = h_j rows), which it masks with the forward's ReLU bits of z
// into da2 (stored positions, as the dz pass does), and the 32-column tile w
// of m_e (as k_dh_u).  dz1 = W2^T da2 and da1 follow in k_da1, whose W2^T
// copy would not fit in LDS beside two U_i.
struct DzDhuArgs {
  DhuArgs m;
  const int32_t* col;
  const unsigned char* h_in;    // [n_src][d] bf16
  const unsigned char* zmask;   // [E][(h1+h2)/8] ReLU mask bits of z1 and z (forward)
  unsigned char* da2E;          // [E][h2] bf16 out, stored positions
};

template <int DL, int H1, int H2>
struct DzDhuShape {
  static constexpr int UB = H2 * DL * 2, GB = DL * 2, BUF = UB + GB, LDS = 2 * BUF;
  static_assert(UB % (256 * 16) == 0 && GB % 16 == 0 && GB / 16 <= 256, "U_i whole rounds, g_i one partial round");
};

template <int DL, int H1, int H2>
__global__ __launch_bounds__(256) void k_dz_dh_u(DzDhuArgs a) {
  using S = DzDhuShape<DL, H1, H2>;
  using M = MT<__bf16>;
  constexpr int SKD = DL / 16, SK2 = H2 / 16, PT = DL / 32, KT = H2 / 32, KTW = KT / 4;
  constexpr int MW1 = H1 / 64, MW2 = H2 / 64, MROW = (H1 + H2) / 8;
  static_assert(PT == 4 && KTW == 2, "one column tile of p and two neuron tiles per wave");
  // two statically distinct buffers: the compiler can then see that the
  // copies into one never alias the reads of the other, and does not wait
  // for the copies before every LDS read
  __shared__ __align__(16) unsigned char XA[S::BUF], XB[S::BUF];
  const DhuArgs& d = a.m;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  bf16x8 ba[SKD];
#pragma unroll
  for (int sf = 0; sf < SKD; ++sf)
    ba[sf] = ld_frag<__bf16>(d.b3n + ((size_t)(32 * wv + l32) * DL + 16 * sf + 8 * hh) * 2);
  // operands of one 32-edge tile: z rows, h_j rows (c: the lane's source) and
  // the mask word of this wave's neurons
  struct Ops {
    bf16x8 z[SK2], h[SKD];
    uint32_t mw;
  };
  auto load_ops = [&](int64_t pa, int64_t pb, int et, int32_t c, Ops& o) {
    const int64_t e = pa + (int64_t)et * 32 + l32;
    const bool valid = e < pb;
    const size_t es = valid ? (size_t)e : 0;
    const unsigned char* zr = d.zE + es * H2 * 2;
#pragma unroll
    for (int s2 = 0; s2 < SK2; ++s2) o.z[s2] = ld_frag_if<__bf16>(zr + (16 * s2 + 8 * hh) * 2, valid);
    const unsigned char* hr = a.h_in + (size_t)(valid ? c : 0) * DL * 2;
#pragma unroll
    for (int s = 0; s < SKD; ++s) o.h[s] = ld_frag_if<__bf16>(hr + (16 * s + 8 * hh) * 2, valid);
    const uint32_t w = reinterpret_cast<const uint32_t*>(a.zmask + es * MROW)[2 * MW1 + hh * MW2 + wv];
    o.mw = valid ? w : 0u;
  };
  auto item = [&](const unsigned char* Xb, int64_t pa, int64_t pb, int et, const Ops& o) {
    const int64_t e = pa + (int64_t)et * 32 + l32;
    f32x16 acc = f32x16{};
    // m_e: the bias row sum_q b3[p*d+q] g_i[q], then the z~ . U_i terms
#pragma unroll
    for (int sf = 0; sf < SKD; ++sf)
      acc = M::mma(ba[sf], *reinterpret_cast<const bf16x8*>(Xb + S::UB + (16 * sf + 8 * hh) * 2), acc);
#pragma unroll
    for (int s2 = 0; s2 < SK2; ++s2) acc = M::mma(lds_frag_ut<DL>(Xb, 16 * s2, 32 * wv), o.z[s2], acc);
    // dz_e on neuron tiles 2w, 2w + 1: fragment (kt, s) of U_i is 64 lanes x 16 bytes
    f32x16 dz[KTW];
#pragma unroll
    for (int kk = 0; kk < KTW; ++kk) {
      dz[kk] = f32x16{};
#pragma unroll
      for (int s = 0; s < SKD; ++s)
        dz[kk] = M::mma(*reinterpret_cast<const bf16x8*>(Xb + (((KTW * wv + kk) * SKD + s) * 64 + lane) * 16),
                        o.h[s], dz[kk]);
    }
    // The tile's only memory operations after the products: eight stores
    // (four of m_e, four of da2).  The next step's wait count relies on it.
    if (e < pb) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const bf16x2 lo = __builtin_convertvector((f32x2){acc[4 * g], acc[4 * g + 1]}, bf16x2);
        const bf16x2 hi = __builtin_convertvector((f32x2){acc[4 * g + 2], acc[4 * g + 3]}, bf16x2);
        *reinterpret_cast<uint2*>(d.mE + ((size_t)e * DL + 32 * wv + 8 * g + 4 * hh) * 2) =
            make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
      }
      // da2 positions 16 s + 8 hh + u, s = 4w + sl, hold dz register 8 (sl % 2) + u of tile sl / 2
#pragma unroll
      for (int sl = 0; sl < 4; ++sl) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = keep_if_bit(dz[sl / 2][8 * (sl % 2) + u], o.mw, 8 * sl + u);
        *reinterpret_cast<bf16x8*>(a.da2E + ((size_t)e * H2 + 16 * (4 * wv + sl) + 8 * hh) * 2) =
            pack_frag<__bf16>(v);
      }
    }
  };
  const int64_t i0 = blockIdx.x, G = gridDim.x;
  if (i0 >= d.n_dst) return;
  // Loads and stores retire through one in-order counter, so waiting for a
  // load also waits for everything issued before it.  Per destination i the
  // order is: the index loads (edge range of i + 3G, first-tile sources of
  // i + 2G), the operand loads of i + G, then the copies of U and g of
  // i + G, then the products of i.  The operand registers are handed on at the
  // end of the step, which waits for those loads but not for the copies
  // behind them; the next step waits for everything (the copies) before its
  // barrier.  Index values are used one step after their loads.
  // edge range of a destination: scalar loads (row_ptr is not written while
  // the kernel runs), which count apart from the vector loads and copies
  typedef __attribute__((address_space(4))) const int32_t cint32_t;
  cint32_t* rp = (cint32_t*)(d.row_ptr);
  auto rows = [&](int64_t i, int64_t& p0, int64_t& p1) {
    const int64_t ic = i < d.n_dst ? i : d.n_dst;
    p0 = rp[ic];
    p1 = i < d.n_dst ? (int64_t)rp[ic + 1] : p0;
  };
  // source of the lane's edge in the first tile of edges [p0, p1) (0 past
  // them; the load is unconditional, of edge 0 there)
  auto first_col = [&](int64_t p0, int64_t p1) -> int32_t {
    const int64_t q = p0 + l32;
    const bool valid = q < p1;
    const int32_t c = a.col[valid ? q : 0];
    return valid ? c : 0;
  };
  int64_t pa, pb, pa1, pb1, pa2, pb2;
  rows(i0, pa, pb);
  rows(i0 + G, pa1, pb1);
  rows(i0 + 2 * G, pa2, pb2);
  Ops opsA, opsB;
  load_ops(pa, pb, 0, first_col(pa, pb), opsA);
  int32_t c1 = first_col(pa1, pb1);
  // U_i is read once, here: streaming copies
  lds_copy_async<LDS_COPY_STREAM>(d.U + (size_t)i0 * S::UB, XA, S::UB / 16);
  lds_copy_async(d.gT + (size_t)i0 * S::GB, XA + S::UB, S::GB / 16);
  // one destination: its U_i and g_i in Xc (copied one step earlier), its
  // operands in cur; the next destination's copies go to Xn, its operands to
  // nxt.  The loop alternates the two (buffers, operand sets) in code, so no
  // buffer is chosen at run time and no operand set is copied.
  int prev_net = 0;   // edge tiles of the previous destination (its stores follow the copies)
  auto step = [&](int64_t i, const unsigned char* Xc, unsigned char* Xn, const Ops& cur, Ops& nxt) {
    // the copies of U_i and g_i: after them the previous step issued only its
    // tile's eight stores when it had one tile, which may stay in flight
    if (prev_net == 1) __builtin_amdgcn_s_waitcnt(vmcnt_imm(8));
    else stage_wait();
    lds_sync();   // U_i, g_i in Xc; every wave is done with Xn (LDS only: stores stay in flight)
    int64_t pa3, pb3;
    rows(i + 3 * G, pa3, pb3);
    const int32_t c2 = first_col(pa2, pb2);
    load_ops(pa1, pb1, 0, c1, nxt);
    {
      // unconditional (the last step copies its own U_i again): the count of
      // operations after the operand loads then includes these copies
      const int64_t inext = i + G < d.n_dst ? i + G : i;
      lds_copy_async<LDS_COPY_STREAM>(d.U + (size_t)inext * S::UB, Xn, S::UB / 16);
      lds_copy_async(d.gT + (size_t)inext * S::GB, Xn + S::UB, S::GB / 16);
    }
    asm volatile("" ::: "memory");   // the copies stay ahead of the tile's stores
    __builtin_amdgcn_sched_barrier(0);
    const int net = (int)((pb - pa + 31) / 32);
    if (net > 0) item(Xc, pa, pb, 0, cur);
    for (int et = 1; et < net; ++et) {   // destinations of more than 32 edges
      const int64_t e = pa + (int64_t)et * 32 + l32;
      const bool valid = e < pb;
      const int32_t c = a.col[valid ? e : pa];
      Ops ox;
      load_ops(pa, pb, et, valid ? c : 0, ox);
      item(Xc, pa, pb, et, ox);
    }
    pa = pa1; pb = pb1;
    pa1 = pa2; pb1 = pb2;
    pa2 = pa3; pb2 = pb3;
    c1 = c2;
    prev_net = net;
  };
  for (int64_t i = i0;;) {
    step(i, XA, XB, opsA, opsB);
    if ((i += G) >= d.n_dst) break;
    step(i, XB, XA, opsB, opsA);
    if ((i += G) >= d.n_dst) break;
  }
}

// dz1 = W2^T da2 and da1 = dz1 * [z1 > 0] for 32-edge tiles of the stored da2
// rows (the second half of the dz epilogue, in the same products and order),
// and the layer-1 weight gradients from them in the same pass:
//   dW1[j][c] = sum_e da1_e[j] x_e[c],  db1[j] = sum_e da1_e[j],
// with x as its bf16 high parts (columns 0..7) and low parts (8..15) next to
// a column of ones (16), as the unfused dW1 product takes it.  W2^T is staged
// in LDS once per workgroup; each wave takes every (4 x grid)-th tile, the
// next tile's da2 rows, mask words and attribute rows loaded while the current
// one is multiplied.  Each 32 x 32 block of da1 goes through a small LDS tile
// of the wave ([edge][stored position]) so that the dW1 product can read it
// with transposing reads (edges are its contraction index); the wave keeps its
// dW1 sums in registers over all its tiles and writes them to partial slot
// 4 blockIdx.x + w.  da1 goes to HBM only when the attribute gradient needs it.
struct Da1Args {
  int64_t E;
  const unsigned char* w2t;     // packed W2^T rows [h1][h2 stored positions] bf16
  const unsigned char* zmask;   // [E][(h1+h2)/8]
  const unsigned char* da2E;    // [E][h2] bf16, stored positions
  const unsigned char* xE;      // [E][32 bytes]: bf16 high parts 0..7, low parts 8..15
  int de;
  unsigned char* da1E;          // [E][h1] bf16 out, or null
  float* p_w1;                  // [4 grid][h1*de + h1] partial sums
};

template <int H1, int H2>
struct Da1Shape {
  static constexpr int W2B = H1 * DzAggShape<__bf16, H1, H2>::W2P;
  static constexpr int TP = 64;                // pitch of the wave's da1 and attribute tiles (bytes)
  static constexpr int WT = 3 * 32 * TP;       // per wave: two da1 tiles, the attribute tile
  static constexpr int LDS = W2B + 4 * WT;
  static_assert(LDS <= 160 * 1024, "LDS of the da1 pass");
};

template <int H1, int H2>
__global__ __launch_bounds__(256) void k_da1_dw1(Da1Args a) {
  using SA = DzAggShape<__bf16, H1, H2>;
  using S = Da1Shape<H1, H2>;
  using M = MT<__bf16>;
  constexpr int SK2 = H2 / 16, JT = H1 / 32, MW1 = H1 / 64, MROW = (H1 + H2) / 8, TP = S::TP;
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  unsigned char* dtile = smem + S::W2B + wv * S::WT;
  unsigned char* xtile = dtile + 2 * 32 * TP;
  {
    LdsStage<H1, H2 * 2> stg;
    stg.init();
    stg.issue(a.w2t, smem);
    // columns 16..31 of the attribute tile: a one in column 16, zeros after it
    const float one[8] = {hh ? 0.0f : 1.0f, 0, 0, 0, 0, 0, 0, 0};
    *reinterpret_cast<bf16x8*>(xtile + l32 * TP + 32 + 16 * hh) = pack_frag<__bf16>(one);
    stage_wait();
    __syncthreads();
  }
  const int64_t ntile = (a.E + 31) / 32, stride = (int64_t)gridDim.x * 4;
  struct Ops {
    bf16x8 B[SK2];
    uint32_t m1[MW1];
    uint4 x;   // bytes 16 hh .. + 15 of the lane's edge's attribute row
  };
  auto load = [&](int64_t t, Ops& o) {   // unconditional loads (row 0 past the edges), then zeroed
    const int64_t e = t * 32 + l32;
    const bool valid = t < ntile && e < a.E;
    const size_t es = valid ? (size_t)e : 0;
#pragma unroll
    for (int s = 0; s < SK2; ++s) o.B[s] = ld_frag_if<__bf16>(a.da2E + (es * H2 + 16 * s + 8 * hh) * 2, valid);
    const uint32_t* mb = reinterpret_cast<const uint32_t*>(a.zmask + es * MROW);
#pragma unroll
    for (int w = 0; w < MW1; ++w) {
      const uint32_t m = mb[hh * MW1 + w];
      o.m1[w] = valid ? m : 0u;
    }
    const uint4 x = *reinterpret_cast<const uint4*>(a.xE + es * 32 + 16 * hh);
    o.x = valid ? x : make_uint4(0, 0, 0, 0);
  };
  f32x16 acc1[JT];
#pragma unroll
  for (int jt = 0; jt < JT; ++jt) acc1[jt] = f32x16{};
  int64_t t = (int64_t)blockIdx.x * 4 + wv;
  Ops o, on;
  load(t, o);
  load(t + stride, on);
  for (; t < ntile; t += stride) {
    // loads run two tiles ahead: one tile's products do not cover their latency
    Ops onn;
    load(t + 2 * stride, onn);
    const int64_t e = t * 32 + l32;
    *reinterpret_cast<uint4*>(xtile + l32 * TP + 16 * hh) = o.x;
    const bf16x8 X0 = lds_frag_rows(xtile, TP, 0, 0), X1 = lds_frag_rows(xtile, TP, 16, 0);
    // two blocks of dz1 at a time, so that two accumulation chains interleave
#pragma unroll
    for (int jp = 0; jp < JT; jp += 2) {
      __builtin_amdgcn_sched_barrier(0);
      f32x16 C[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int s = 0; s < SK2; ++s) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const bf16x8 A =
              *reinterpret_cast<const bf16x8*>(smem + ((jp + q) * 32 + l32) * SA::W2P + (16 * s + 8 * hh) * 2);
          C[q] = M::mma(A, o.B[s], C[q]);
        }
      }
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int jt = jp + q;
        unsigned char* dt = dtile + q * 32 * TP;
        // register i of block jt is stored position 16 (2 jt + i / 8) + 8 hh + i % 8
#pragma unroll
        for (int i = 0; i < 16; i += 8) {
          const int n = 16 * jt + i;
          float v[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) v[u] = keep_if_bit(C[q][i + u], o.m1[(n + u) / 32], (n + u) % 32);
          const bf16x8 f = pack_frag<__bf16>(v);
          if (a.da1E && e < a.E)
            *reinterpret_cast<bf16x8*>(a.da1E + ((size_t)e * H1 + (n / 8) * 16 + 8 * hh) * 2) = f;
          *reinterpret_cast<bf16x8*>(dt + l32 * TP + (16 * (i / 8) + 8 * hh) * 2) = f;
        }
        // dW1 rows of this block: A = da1 [position][edge], B = the attribute columns
        acc1[jt] = M::mma(lds_frag_rows(dt, TP, 0, 0), X0, acc1[jt]);
        acc1[jt] = M::mma(lds_frag_rows(dt, TP, 16, 0), X1, acc1[jt]);
      }
    }
    o = on;
    on = onn;
  }
  // column c of a block holds the high-part sums, column c + 8 the low-part
  // sums, column 16 the row sums (db1)
  float* out = a.p_w1 + (size_t)(blockIdx.x * 4 + wv) * (H1 * a.de + H1);
#pragma unroll
  for (int jt = 0; jt < JT; ++jt) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float lo = __shfl_down(acc1[jt][i], 8, 64);
      const int j = kperm<__bf16>(jt * 32 + 8 * (i / 4) + 4 * hh + (i % 4));
      if (l32 < a.de) out[(size_t)j * a.de + l32] = acc1[jt][i] + lo;
      if (l32 == 16) out[(size_t)H1 * a.de + j] = acc1[jt][i];
    }
  }
}

template <int DL, int H2>
dsmp_status launch_dh_u(dsmp_handle* h, const DhuArgs& a) {
  using S = DhuShape<DL, H2>;
  auto k = k_dh_u<DL, H2>;
  DSMP_HIP(h, hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                  S::LDS));
  int per_cu = 0;
  DSMP_HIP(h, hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, 256, S::LDS));
  const int64_t grid = std::min<int64_t>(a.n_dst, (int64_t)h->n_cu * std::max(per_cu, 1));
  if (grid == 0) return DSMP_OK;
  hipLaunchKernelGGL(k, dim3((unsigned)grid), dim3(256), S::LDS, h->stream, a);
  DSMP_LAUNCHED(h, "feature gradient from U");
  return DSMP_OK;
}

dsmp_status dispatch_dh_u(dsmp_handle* h, const dsmp_layer_desc& d, const DhuArgs& a) {
  if (d.d == 32 && d.h2 == 64) return launch_dh_u<32, 64>(h, a);
  if (d.d == 32 && d.h2 == 128) return launch_dh_u<32, 128>(h, a);
  if (d.d == 64 && d.h2 == 64) return launch_dh_u<64, 64>(h, a);
  if (d.d == 64 && d.h2 == 128) return launch_dh_u<64, 128>(h, a);
  if (d.d == 128 && d.h2 == 256) return launch_dh_u<128, 256>(h, a);
  return fail(h, DSMP_UNSUPPORTED, "unsupported layer shape for the feature gradient from U");
}

// The feature gradient comes from U (and no per-source sums are formed) for
// bf16 layers of the aggregate form.
bool dh_from_u(const dsmp_layer_desc& d, bool agg) { return agg && d.dtype == DSMP_BF16; }




// ------------------------------------------------------------ workspace

struct BwdWs {
  float *gF, *dh_node, *dh_direct, *dh_part, *dh_sl;
  unsigned char *gT, *da2E, *da1E, *ot, *U, *mE;
  float4* dx;                  // [E] edge-attribute gradients (diff attributes)
  int nslh;
  float *p_root, *p_db3, *p_w3, *p_w2, *p_w1;
  int nr, nb3, n3, n2, n1;
  int64_t pc3, pc2, pc1, pr, pb3;
  size_t total;
};

int w3_pb(int d, int h2) {
  const int qt = d / 32, kt = h2 / 32, ktw = kt < 4 ? kt : 4;
  const bool pair = qt * (kt / ktw) <= 2;
  const int qtw = pair ? 1 : 2, pw = pair ? 2 : 1, wpg = (qt / qtw) * (kt / ktw);
  return (4 / wpg) * pw;
}

int w3_nchunk(int d, int h2, int64_t E) {
  int npb = d / w3_pb(d, h2);
  int target = 1024 / npb;
  int n = ((target + 7) / 8) * 8;
  if (n < 8) n = 8;
  int64_t maxn = ((E + 63) / 64 + 7) / 8 * 8;
  if (maxn < 8) maxn = 8;
  if (n > maxn) n = (int)maxn;
  return n;
}

BwdWs carve_bwd(const dsmp_layer_desc& d, int64_t n_dst, int64_t n_src, int64_t E, void* base) {
  Carve c(base);
  BwdWs w;
  const int esz = d.dtype == DSMP_BF16 ? 2 : 4;
  const int de = layer_attr_width(d);
  w.gF = c.take<float>((size_t)n_dst * d.d);
  w.gT = c.take<unsigned char>((size_t)n_dst * d.d * esz);
  w.dh_node = c.take<float>((size_t)n_dst * d.d);
  w.dh_direct = c.take<float>((size_t)n_src * d.d);
  w.dh_part = c.take<float>((size_t)(ceil_div(E, EDGE_TILE) + 1) * 2 * d.d);
  // aggregate form: per-source sums T and the K-slices of their W3 GEMM
  w.ot = c.take<unsigned char>((size_t)n_src * agg_ktot(d) * esz + 256);   // + whole last staged piece
  w.nslh = agg_gemm_slices(n_src, d);
  w.dh_sl = c.take<float>((size_t)w.nslh * n_src * d.d);
  w.U = c.take<unsigned char>((size_t)n_dst * d.h2 * d.d * esz);
  w.mE = c.take<unsigned char>((size_t)E * d.d * esz);   // per-edge feature-gradient terms (from U)
  w.da2E = c.take<unsigned char>((size_t)E * d.h2 * esz);
  w.da1E = c.take<unsigned char>((size_t)E * d.h1 * esz);
  w.dx = c.take<float4>((size_t)E);
  w.nr = (int)(n_dst > 0 ? (ceil_div(n_dst, 32) < 1024 ? ceil_div(n_dst, 32) : 1024) : 1);
  w.pr = n_dst > 0 ? ceil_div(n_dst, w.nr) : 1;
  w.p_root = c.take<float>((size_t)w.nr * (d.d * d.d + d.d));
  w.nb3 = w.nr;
  w.pb3 = w.pr;
  w.p_db3 = c.take<float>((size_t)w.nb3 * d.d * d.d);
  w.n3 = w3_nchunk(d.d, d.h2, E);
  w.pc3 = ((E + w.n3 - 1) / w.n3 + 63) / 64 * 64;
  if (w.pc3 < 64) w.pc3 = 64;
  // dW3 partials: per-edge chunks, or the node slices of the aggregate form
  const size_t p3e = (size_t)w.n3 * d.d * d.d * d.h2;
  const size_t p3a = (size_t)agg_dw3_slices(n_dst) * d.d * agg_ktot(d);
  w.p_w3 = c.take<float>(p3e > p3a ? p3e : p3a);
  // edge chunks of the dW2 and dW1 partial sums: 64 edges or more each, at
  // most 512 (dW2) and 2048 (dW1) chunks, so that small graphs still spread
  // over the CUs
  w.n2 = (int)(E > 0 ? (ceil_div(E, 64) < 512 ? ceil_div(E, 64) : 512) : 1);
  w.pc2 = ((E + w.n2 - 1) / w.n2 + 63) / 64 * 64;
  if (w.pc2 < 64) w.pc2 = 64;
  w.p_w2 = c.take<float>((size_t)w.n2 * (d.h2 * d.h1 + d.h2));
  w.n1 = (int)(E > 0 ? (ceil_div(E, 64) < 2048 ? ceil_div(E, 64) : 2048) : 1);
  w.pc1 = E > 0 ? (E + w.n1 - 1) / w.n1 : 1;
  w.p_w1 = c.take<float>((size_t)w.n1 * (d.h1 * de + d.h1));
  w.total = c.used();
  return w;
}

template <typename K>
dsmp_status set_lds(dsmp_handle* h, K kernel, int bytes) {
  DSMP_HIP(h, hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, bytes));
  return DSMP_OK;
}

template <typename T, int DL, int H1, int H2>
dsmp_status run_edge_grads(dsmp_handle* h, const DzArgs& dz, const W3Args& w3, const W2Args& w2,
                           const DzDhuArgs* fm, Da1Args* fa, int n1cap, int* n1_used) {
  hipStream_t s = h->stream;
  dsmp_status st;
  if (dz.E > 0 && dz.U) {
    // aggregate form: U = g W3 for every destination, then the masked per-tile products
    {
      ProfScope prof(h, DSMP_K_U_GEMM);
      UArgs ua{dz.n_dst, dz.gT, dz.packed + dz.L.w3u, const_cast<unsigned char*>(dz.U)};
      if ((st = launch_u_gemm<T, DL, H2>(h, ua)) != DSMP_OK) return st;
    }
    if (fm) {
      if constexpr (sizeof(T) == 2 && DL == 128 && H1 == 256 && H2 == 256) {
        {
          // dz (masked into da2) and the feature-gradient terms from one read of U
          auto kf = k_dz_dh_u<DL, H1, H2>;   // static LDS: two U_i + g_i buffers
          int per_cu = 0;
          DSMP_HIP(h, hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kf, 256, 0));
          const int64_t grid = std::min<int64_t>(dz.n_dst, (int64_t)h->n_cu * std::max(per_cu, 1));
          ProfScope prof(h, DSMP_K_DZ);
          if (grid > 0) hipLaunchKernelGGL(kf, dim3((unsigned)grid), dim3(256), 0, s, *fm);
          DSMP_LAUNCHED(h, "dz and feature-gradient terms from U");
        }
        {
          // da1 and the dW1/db1 partial sums (four per workgroup, at most n1cap)
          using SD = Da1Shape<H1, H2>;
          auto ka = k_da1_dw1<H1, H2>;
          if ((st = set_lds(h, ka, SD::LDS)) != DSMP_OK) return st;
          int per_cu = 0;
          DSMP_HIP(h, hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, ka, 256, SD::LDS));
          int64_t grid = std::min<int64_t>(ceil_div(ceil_div(dz.E, 32), 4), (int64_t)h->n_cu * std::max(per_cu, 1));
          grid = std::max<int64_t>(1, std::min<int64_t>(grid, n1cap / 4));
          ProfScope prof(h, DSMP_K_DA1);
          hipLaunchKernelGGL(ka, dim3((unsigned)grid), dim3(256), SD::LDS, s, *fa);
          DSMP_LAUNCHED(h, "da1 and dW1 from da2");
          *n1_used = (int)(4 * grid);
        }
      } else {
        return fail(h, DSMP_UNSUPPORTED, "dz with the feature-gradient terms is built for d = 128, h = 256 only");
      }
    } else {
    using SA = DzAggShape<T, H1, H2>;
    auto kz = k_bwd_dz_agg<T, DL, H1, H2>;
    if ((st = set_lds(h, kz, SA::LDS)) != DSMP_OK) return st;
    int per_cu = 0;
    DSMP_HIP(h, hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kz, 256, SA::LDS));
    // blocks of up to DZ_NB destinations, smaller where that leaves CUs idle
    const int64_t slots = (int64_t)h->n_cu * std::max(per_cu, 1);
    DzArgs da = dz;
    da.nb = (int)std::max<int64_t>(1, std::min<int64_t>(DZ_NB, ceil_div(dz.n_dst, slots)));
    const int64_t grid = std::min<int64_t>(ceil_div(dz.n_dst, da.nb), slots);
    ProfScope prof(h, DSMP_K_DZ);
    hipLaunchKernelGGL(kz, dim3((unsigned)grid), dim3(256), SA::LDS, s, da);
    DSMP_LAUNCHED(h, "dz (aggregate form)");
    }
  } else if (dz.E > 0) {
    using S = DzShape<T, DL, H1, H2>;
    auto kz = k_bwd_dz<T, DL, H1, H2>;
    if ((st = set_lds(h, kz, S::LDS)) != DSMP_OK) return st;
    ProfScope prof(h, DSMP_K_DZ);
    hipLaunchKernelGGL(kz, dim3(ceil_div(dz.E, S::TILE)), dim3(256), S::LDS, s, dz);
    DSMP_LAUNCHED(h, "dz");
  }
  if (w3.nchunk > 0) {
    using S = W3Shape<T, DL, H2>;
    auto k3 = k_bwd_dW3<T, DL, H2>;
    if ((st = set_lds(h, k3, S::LDS)) != DSMP_OK) return st;
    ProfScope prof(h, DSMP_K_DW3);
    hipLaunchKernelGGL(k3, dim3((DL / S::PB) * w3.nchunk), dim3(256), S::LDS, s, w3);
    DSMP_LAUNCHED(h, "dW3");
  }
  {
    using S = W2Shape<T, H1, H2>;
    int nchunk = (int)((w2.E + w2.per_chunk - 1) / w2.per_chunk);
    if (nchunk < 1) nchunk = 1;
    if constexpr (sizeof(T) == 2) {
      using TS = W2TrShape<H1, H2>;
      if constexpr (S::NSPLIT > 1 && H1 == 256 && H2 == 256) {
        if (w2.z1E == nullptr) {   // z1 recomputed from the split attributes
          auto k2 = k_bwd_dW2_rz<H1, H2>;
          ProfScope prof(h, DSMP_K_DW2);
          hipLaunchKernelGGL(k2, dim3(nchunk), dim3(512), 0, s, w2);
        } else {
          auto k2 = k_bwd_dW2_tr<H1, H2, true>;
          if ((st = set_lds(h, k2, TS::LDS)) != DSMP_OK) return st;
          ProfScope prof(h, DSMP_K_DW2);
          hipLaunchKernelGGL(k2, dim3(nchunk), dim3(512), TS::LDS, s, w2);
        }
      } else {
        auto k2 = k_bwd_dW2_tr<H1, H2>;
        if ((st = set_lds(h, k2, TS::LDS)) != DSMP_OK) return st;
        ProfScope prof(h, DSMP_K_DW2);
        hipLaunchKernelGGL(k2, dim3(nchunk * S::NSPLIT), dim3(256), TS::LDS, s, w2);
      }
    } else {
      auto k2 = k_bwd_dW2<T, H1, H2>;
      if ((st = set_lds(h, k2, S::LDS)) != DSMP_OK) return st;
      ProfScope prof(h, DSMP_K_DW2);
      hipLaunchKernelGGL(k2, dim3(nchunk * S::NSPLIT), dim3(256), S::LDS, s, w2);
    }
    DSMP_LAUNCHED(h, "dW2");
  }
  return DSMP_OK;
}

template <int H1>
dsmp_status launch_dw1_tr(dsmp_handle* h, int n1, int64_t E, int64_t pc1, const unsigned char* da1E,
                          const unsigned char* xE, int de, float* part) {
  using S = W1TrShape<H1>;
  auto k1 = k_bwd_dW1_tr<H1>;
  dsmp_status st = set_lds(h, k1, S::LDS);
  if (st != DSMP_OK) return st;
  hipLaunchKernelGGL(k1, dim3(n1), dim3(256), S::LDS, h->stream, E, pc1, da1E, xE, de, part);
  return DSMP_OK;
}

dsmp_status dispatch_edge_grads(dsmp_handle* h, const dsmp_layer_desc& d, const DzArgs& dz, const W3Args& w3,
                                const W2Args& w2, const DzDhuArgs* fm, Da1Args* fa, int n1cap, int* n1_used) {
  if (d.dtype == DSMP_F32) {
    if (d.d == 32) return run_edge_grads<float, 32, 64, 64>(h, dz, w3, w2, fm, fa, n1cap, n1_used);
    if (d.d == 64) return run_edge_grads<float, 64, 128, 128>(h, dz, w3, w2, fm, fa, n1cap, n1_used);
  } else {
    if (d.d == 32) return run_edge_grads<__bf16, 32, 64, 64>(h, dz, w3, w2, fm, fa, n1cap, n1_used);
    if (d.d == 64) return run_edge_grads<__bf16, 64, 128, 128>(h, dz, w3, w2, fm, fa, n1cap, n1_used);
    if (d.d == 128) return run_edge_grads<__bf16, 128, 256, 256>(h, dz, w3, w2, fm, fa, n1cap, n1_used);
  }
  return fail(h, DSMP_UNSUPPORTED, "unsupported layer shape");
}

// Aggregate form, bf16, h1 = h2 <= 128: U = g W3 for every destination, then
// one fused pass for dz, da2, da1 and the dW2/db2/dW1/db1 partial sums
// (one partial per workgroup, at most cap workgroups).
template <int DL, int H1, int H2>
dsmp_status run_edge_grads_fused(dsmp_handle* h, const EdgeGradArgs& eg, int cap, int* nchunk) {
  hipStream_t s = h->stream;
  const DzArgs& dz = eg.dz;
  {
    ProfScope prof(h, DSMP_K_U_GEMM);
    UArgs ua{dz.n_dst, dz.gT, dz.packed + dz.L.w3u, const_cast<unsigned char*>(dz.U)};
    dsmp_status su = launch_u_gemm<__bf16, DL, H2>(h, ua);
    if (su != DSMP_OK) return su;
  }
  using G = EdgeGradShape<DL, H1, H2>;
  auto kf = k_bwd_edge_agg<DL, H1, H2>;
  dsmp_status st = set_lds(h, kf, G::LDS);
  if (st != DSMP_OK) return st;
  int per_cu = 0;
  DSMP_HIP(h, hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kf, G::NT, G::LDS));
  int64_t grid = std::min<int64_t>((dz.n_dst + DZ_NB - 1) / DZ_NB, (int64_t)h->n_cu * std::max(per_cu, 1));
  grid = std::max<int64_t>(1, std::min<int64_t>(grid, cap));
  ProfScope prof(h, DSMP_K_DZ);
  hipLaunchKernelGGL(kf, dim3((unsigned)grid), dim3(G::NT), G::LDS, s, eg);
  DSMP_LAUNCHED(h, "fused edge gradients");
  *nchunk = (int)grid;
  return DSMP_OK;
}

dsmp_status dispatch_edge_grads_fused(dsmp_handle* h, const dsmp_layer_desc& d, const EdgeGradArgs& eg, int cap,
                                      int* nchunk) {
  if (d.d == 32 && d.h1 == 64) return run_edge_grads_fused<32, 64, 64>(h, eg, cap, nchunk);
  if (d.d == 64 && d.h1 == 64) return run_edge_grads_fused<64, 64, 64>(h, eg, cap, nchunk);
  if (d.d == 32 && d.h1 == 128) return run_edge_grads_fused<32, 128, 128>(h, eg, cap, nchunk);
  if (d.d == 64 && d.h1 == 128) return run_edge_grads_fused<64, 128, 128>(h, eg, cap, nchunk);
  return fail(h, DSMP_UNSUPPORTED, "unsupported layer shape for the fused edge gradients");
}

template <typename T, int DL>
void launch_node_kernels(dsmp_handle* h, const BNodeArgs& na, int64_t n_dst, const BwdWs& w,
                         const unsigned char* h_in, const int32_t* row_ptr, const int32_t* col, bool db3) {
  hipStream_t s = h->stream;
  if (n_dst == 0) return;
  if constexpr (std::is_same<T, __bf16>::value && DL == 64)
    hipLaunchKernelGGL((k_bwd_node_m<64, 4>), dim3(w.nr), dim3(256), 0, s, na);
  else if constexpr (std::is_same<T, __bf16>::value && DL == 128)
    hipLaunchKernelGGL((k_bwd_node_m<128, 8>), dim3(w.nr), dim3(512), 0, s, na);
  else
    hipLaunchKernelGGL((k_bwd_node<T, DL>), dim3(w.nr), dim3(256), 0, s, na);
  if (db3)
    hipLaunchKernelGGL((k_bwd_db3<T, DL>), dim3(w.nb3), dim3(256), 0, s, n_dst, w.pb3, row_ptr, col, h_in, w.gF,
                       w.p_db3);
}

}  // namespace

namespace dsmp {
// Where the kernel-MLP gradients are not fused (bf16, d = 128, h1 = h2 = 256)
// the dz pass also forms the feature-gradient terms (k_dz_dh_u), the da1 pass
// the dW1 sums, and the dW2 pass recomputes z1 (the forward keeps no z1 rows).
bool dz_with_m(const dsmp_layer_desc& d, bool agg) {
  return agg && d.dtype == DSMP_BF16 && d.d == 128 && d.h1 == 256 && d.h2 == 256;
}

bool fused_edge_grads(const dsmp_layer_desc& d) {
  return d.dtype == DSMP_BF16 && d.h1 == d.h2 && (d.h1 == 64 || d.h1 == 128) && (d.d == 32 || d.d == 64);
}
}  // namespace dsmp

extern "C" dsmp_status dsmp_nnconv_workspace(const dsmp_layer_desc* desc, const dsmp_graph* g,
                                             size_t* saved_bytes, size_t* fwd_ws, size_t* bwd_ws) {
  if (!desc || !g || !saved_bytes || !fwd_ws || !bwd_ws) return DSMP_INVALID_ARG;
  dsmp_status st = check_layer_desc(nullptr, desc);
  if (st != DSMP_OK) return st;
  if (g->n_dst < 0 || g->n_src < g->n_dst || g->n_edges < 0) return DSMP_INVALID_ARG;
  *saved_bytes = saved_layout(*desc, g->n_dst, g->n_edges).total;
  *fwd_ws = fwd_ws_bytes(*desc, g->n_dst, g->n_edges);
  *bwd_ws = carve_bwd(*desc, g->n_dst, g->n_src, g->n_edges, nullptr).total;
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_nnconv_backward(dsmp_handle* h, const dsmp_layer_desc* desc, const void* packed,
                                            const dsmp_graph* g, const float* node_attr, const void* h_in,
                                            const void* saved, size_t saved_bytes, const float* grad_out,
                                            float* grad_h, const dsmp_layer_grads* grads, int32_t flags, void* ws,
                                            size_t ws_bytes) {
  if (!h) return DSMP_INVALID_ARG;
  dsmp_status st = check_layer_desc(h, desc);
  if (st != DSMP_OK) return st;
  if ((st = check_graph(h, g, true)) != DSMP_OK) return st;
  const dsmp_layer_desc& d = *desc;
  DSMP_CHECK(h, packed && saved && grads, DSMP_INVALID_ARG, "packed, saved or grads is NULL");
  DSMP_CHECK(h, grads->dW1 && grads->db1 && grads->dW2 && grads->db2 && grads->dW3 && grads->db3 && grads->dWr &&
                    grads->dbr, DSMP_INVALID_ARG, "a gradient pointer is NULL");
  DSMP_CHECK(h, (g->n_dst == 0 || grad_out) && (g->n_src == 0 || (grad_h && h_in && node_attr)),
             DSMP_INVALID_ARG, "a backward pointer is NULL");
  DSMP_CHECK(h, (flags & ~(DSMP_GRAD_ACCUMULATE | DSMP_GRAD_X_ACCUMULATE)) == 0, DSMP_INVALID_ARG, "unknown flags");
  DSMP_CHECK(h, !grads->dattr || desc->attr_mode == DSMP_ATTR_DIFF, DSMP_UNSUPPORTED,
             "the attribute gradient needs difference edge attributes");
  const SavedLayout sl = saved_layout(d, g->n_dst, g->n_edges);
  DSMP_CHECK(h, saved_bytes >= sl.total, DSMP_WORKSPACE_TOO_SMALL, "saved buffer needs %zu bytes", sl.total);
  const BwdWs need = carve_bwd(d, g->n_dst, g->n_src, g->n_edges, nullptr);
  DSMP_CHECK(h, ws && ws_bytes >= need.total, DSMP_WORKSPACE_TOO_SMALL, "backward workspace needs %zu bytes",
             need.total);
  const BwdWs w = carve_bwd(d, g->n_dst, g->n_src, g->n_edges, ws);
  const int esz = d.dtype == DSMP_BF16 ? 2 : 4;
  const int de = layer_attr_width(d);
  const PackLayout L = pack_layout(d.d, d.h1, d.h2, esz);
  const unsigned char* pk = static_cast<const unsigned char*>(packed);
  const unsigned char* sv = static_cast<const unsigned char*>(saved);
  const unsigned char* hin = static_cast<const unsigned char*>(h_in);
  hipStream_t s = h->stream;
  const int acc = flags & DSMP_GRAD_ACCUMULATE;
  const int64_t E = g->n_edges, n_dst = g->n_dst, n_src = g->n_src;

  const bool agg = use_aggregate(h, d, n_dst, E);

  // node pre-pass, root grads, db3 partials (the aggregate form takes db3
  // from the bias rows of its dW3 product)
  ProfScope prof_node(h, DSMP_K_NODE_BWD);
  BNodeArgs na{n_dst, w.pr, g->row_ptr, grad_out, reinterpret_cast<const float*>(sv + sl.y),
               reinterpret_cast<const float*>(pk + L.wr), hin, w.gT, w.gF, w.dh_node, w.p_root, d.act, d.residual};
  if (d.dtype == DSMP_BF16) {
    if (d.d == 32) launch_node_kernels<__bf16, 32>(h, na, n_dst, w, hin, g->row_ptr, g->col, !agg);
    if (d.d == 64) launch_node_kernels<__bf16, 64>(h, na, n_dst, w, hin, g->row_ptr, g->col, !agg);
    if (d.d == 128) launch_node_kernels<__bf16, 128>(h, na, n_dst, w, hin, g->row_ptr, g->col, !agg);
  } else {
    if (d.d == 32) launch_node_kernels<float, 32>(h, na, n_dst, w, hin, g->row_ptr, g->col, !agg);
    if (d.d == 64) launch_node_kernels<float, 64>(h, na, n_dst, w, hin, g->row_ptr, g->col, !agg);
  }
  DSMP_LAUNCHED(h, "backward node kernels");
  prof_node.end();

  // feature gradient through the edges (edge contraction in source order)
  EdgeArgs ea{};
  ea.E = E; ea.n_dst = n_dst; ea.n_src = n_src;
  ea.row_ptr = g->row_ptr; ea.col = g->col; ea.dst = g->dst; ea.csc_ptr = g->csc_ptr; ea.csc_eid = g->csc_eid;
  ea.node_attr = node_attr; ea.dim = d.dim; ea.attr_mode = d.attr_mode;
  ea.gath = w.gT; ea.packed = pk; ea.L = L;
  ea.zE = const_cast<unsigned char*>(sv + sl.zE);
  ea.z1E = nullptr;
  ea.out_direct = w.dh_direct; ea.out_part = w.dh_part;
  const bool dhu = dh_from_u(d, agg), dzm = dz_with_m(d, agg);
  if (dhu) {
    // after the kernel-MLP gradients, from U (below)
  } else if (agg) {
    // per-source sums T_j = sum_e [z_e; 1] (x) g_e, then one GEMM with W3~
    {
      ProfScope prof(h, DSMP_K_OUTER_DH);
      st = launch_outer_sum(h, d, n_src, g->csc_ptr, g->csc_eid, g->dst, sv + sl.zE, w.gT, w.ot);
    }
    if (st != DSMP_OK) return st;
    {
      ProfScope prof(h, DSMP_K_GEMM_DH);
      st = launch_w3_gemm(h, d, n_src, w.ot, pk + L.wht, w.nslh, w.dh_sl);
    }
    if (st != DSMP_OK) return st;
  } else {
    if ((st = launch_edge_contract(h, d, MODE_DH, ea)) != DSMP_OK) return st;
  }
  if (n_src > 0 && !dhu) {
    unsigned grid = ceil_div(n_src * d.d, 256);
    if (grid > 4096) grid = 4096;
    ProfScope prof(h, DSMP_K_DH_FINAL);
    hipLaunchKernelGGL(k_bwd_dh_final, dim3(grid), dim3(256), 0, s, n_src, n_dst, d.d, g->csc_ptr, w.dh_direct,
                       w.dh_part, agg ? w.nslh : 0, w.dh_sl, w.dh_node, grad_h);
    DSMP_LAUNCHED(h, "grad_h");
  }

  // kernel-MLP gradients
  int nfused = 0;   // workgroups of the fused edge-gradient pass (their partials replace dW2's and dW1's)
  int n1da = 0;     // dW1 partials of the da1 pass (dz_with_m)
  if (E > 0 && agg && fused_edge_grads(d)) {
    DzArgs dz{E, g->col, g->dst, hin, w.gF, pk, L, sv + sl.zE, sv + sl.zmask, w.da2E, w.da1E,
              w.U, w.gT, n_dst, g->row_ptr};
    EdgeGradArgs eg{dz, node_attr, d.dim, d.attr_mode, de, grads->dattr ? w.da1E : nullptr, w.p_w2, w.p_w1};
    if ((st = dispatch_edge_grads_fused(h, d, eg, std::min(w.n2, w.n1), &nfused)) != DSMP_OK) return st;
  } else if (E > 0) {
    DzArgs dz{E, g->col, g->dst, hin, w.gF, pk, L, sv + sl.zE, sv + sl.zmask, w.da2E, w.da1E,
              agg ? w.U : nullptr, w.gT, n_dst, g->row_ptr};
    W3Args w3{E, w.pc3, agg ? 0 : w.n3, g->col, g->dst, hin, w.gF, sv + sl.zE, w.p_w3};
    W2Args w2{E, w.pc2, 1, w.da2E, dzm ? nullptr : sv + sl.z1E, w.p_w2, sv + sl.xE, pk + L.w1l, pk + L.b1l};
    DzDhuArgs fm{DhuArgs{n_dst, g->row_ptr, w.U, w.gT, pk + L.b3n, sv + sl.zE, w.mE}, g->col, hin, sv + sl.zmask,
                 w.da2E};
    Da1Args fa{E, pk + L.w2t, sv + sl.zmask, w.da2E, sv + sl.xE, de, grads->dattr ? w.da1E : nullptr, w.p_w1};
    if ((st = dispatch_edge_grads(h, d, dz, w3, w2, dzm ? &fm : nullptr, &fa, w.n1, &n1da)) != DSMP_OK) return st;
    if (!dzm) {   // with dz_with_m the da1 pass formed the dW1 partial sums
    int n1 = (int)((E + w.pc1 - 1) / w.pc1);
    ProfScope prof(h, DSMP_K_DW1);
    const float* da1f = reinterpret_cast<const float*>(w.da1E);
    if (d.dtype == DSMP_F32 && d.h1 == 64)
      hipLaunchKernelGGL((k_bwd_dW1<float, 64>), dim3(n1), dim3(256), 0, s, E, w.pc1, g->col, g->dst, node_attr,
                         d.dim, d.attr_mode, de, da1f, w.p_w1);
    else if (d.dtype == DSMP_F32)
      hipLaunchKernelGGL((k_bwd_dW1<float, 128>), dim3(n1), dim3(256), 0, s, E, w.pc1, g->col, g->dst, node_attr,
                         d.dim, d.attr_mode, de, da1f, w.p_w1);
    else if (d.h1 == 64)
      st = launch_dw1_tr<64>(h, n1, E, w.pc1, w.da1E, sv + sl.xE, de, w.p_w1);
    else if (d.h1 == 128)
      st = launch_dw1_tr<128>(h, n1, E, w.pc1, w.da1E, sv + sl.xE, de, w.p_w1);
    else
      st = launch_dw1_tr<256>(h, n1, E, w.pc1, w.da1E, sv + sl.xE, de, w.p_w1);
    if (st != DSMP_OK) return st;
    DSMP_LAUNCHED(h, "dW1");
    }
  }

  if (dhu) {
    if (E > 0 && !dzm) {
      ProfScope prof(h, DSMP_K_DH_U);
      DhuArgs da{n_dst, g->row_ptr, w.U, w.gT, pk + L.b3n, sv + sl.zE, w.mE};
      if ((st = dispatch_dh_u(h, d, da)) != DSMP_OK) return st;
    }
    if (n_src > 0) {
      unsigned grid = ceil_div(n_src, 4);
      if (grid > 8192) grid = 8192;
      ProfScope prof(h, DSMP_K_DH_FINAL);
      auto kg = d.d == 32 ? k_dh_gather<32> : d.d == 64 ? k_dh_gather<64> : k_dh_gather<128>;
      hipLaunchKernelGGL(kg, dim3(grid), dim3(256), 0, s, n_src, n_dst, g->csc_ptr, g->csc_eid, w.mE, w.dh_node,
                         grad_h);
      DSMP_LAUNCHED(h, "grad_h from the edge terms");
    }
  }

  if (grads->dattr && n_src > 0) {
    // node-attribute gradient through the difference edge attributes
    ProfScope prof(h, DSMP_K_ATTR);
    if (E > 0) {
      const float* w1l = reinterpret_cast<const float*>(pk + L.w1l);
      if (d.dtype == DSMP_BF16)
        st = d.h1 == 64 ? launch_attr_dx<__bf16, 64>(h, E, w.da1E, w1l, w.dx)
             : d.h1 == 128 ? launch_attr_dx<__bf16, 128>(h, E, w.da1E, w1l, w.dx)
                           : launch_attr_dx<__bf16, 256>(h, E, w.da1E, w1l, w.dx);
      else
        st = d.h1 == 64 ? launch_attr_dx<float, 64>(h, E, w.da1E, w1l, w.dx)
                        : launch_attr_dx<float, 128>(h, E, w.da1E, w1l, w.dx);
      if (st != DSMP_OK) return st;
    }
    hipLaunchKernelGGL(k_attr_seg, dim3(ceil_div(n_src * 16, 256)), dim3(256), 0, s, n_src, n_dst, de, g->row_ptr,
                       g->csc_ptr, g->csc_eid, w.dx, grads->dattr, (flags & DSMP_GRAD_X_ACCUMULATE) ? 1 : 0);
    DSMP_LAUNCHED(h, "attribute gradient sums");
  }

  if (agg) {
    // dW3[p*d+q][k] = sum_i g_i[q] S_i[k][p] from the forward's sums
    ProfScope prof(h, DSMP_K_DW3);
    if ((st = launch_dw3_agg(h, d, n_dst, sv + sl.os, w.gT, w.p_w3, grads->dW3, grads->db3, acc)) != DSMP_OK)
      return st;
  }

  // fixed-order reductions into the caller's gradients, one launch
  RedArgs ra{};
  ra.accumulate = acc;
  auto red = [&](const float* part, int nchunk, int64_t stride, int64_t off, int64_t n, float* out) {
    if (n == 0) return;
    ra.seg[ra.nseg] = RedSeg{part, out, stride, off, n, nchunk};
    ra.first[ra.nseg + 1] = ra.first[ra.nseg] + ceil_div(n, 64);
    ++ra.nseg;
  };
  const int64_t dd = (int64_t)d.d * d.d;
  const int n3 = E > 0 && !agg ? w.n3 : 0;
  const int n2 = nfused ? nfused : E > 0 ? (int)((E + w.pc2 - 1) / w.pc2) : 0;
  const int n1 = nfused ? nfused : n1da ? n1da : E > 0 ? (int)((E + w.pc1 - 1) / w.pc1) : 0;
  const int nr = n_dst > 0 ? w.nr : 0;
  ProfScope prof_red(h, DSMP_K_REDUCE);
  red(w.p_root, nr, dd + d.d, 0, dd, grads->dWr);
  red(w.p_root, nr, dd + d.d, dd, d.d, grads->dbr);
  if (!agg) red(w.p_db3, nr, dd, 0, dd, grads->db3);
  if (!agg) red(w.p_w3, n3, dd * d.h2, 0, dd * d.h2, grads->dW3);
  red(w.p_w2, n2, (int64_t)d.h2 * d.h1 + d.h2, 0, (int64_t)d.h2 * d.h1, grads->dW2);
  red(w.p_w2, n2, (int64_t)d.h2 * d.h1 + d.h2, (int64_t)d.h2 * d.h1, d.h2, grads->db2);
  red(w.p_w1, n1, (int64_t)d.h1 * de + d.h1, 0, (int64_t)d.h1 * de, grads->dW1);
  red(w.p_w1, n1, (int64_t)d.h1 * de + d.h1, (int64_t)d.h1 * de, d.h1, grads->db1);
  if (ra.nseg > 0)
    hipLaunchKernelGGL(k_reduce_multi, dim3((unsigned)ra.first[ra.nseg]), dim3(64 * RED_GROUPS), 0, s, ra);
  DSMP_LAUNCHED(h, "gradient reductions");
  return DSMP_OK;
}
