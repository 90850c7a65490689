// Node-wise networks and loss of the hop loop (Algorithm 1): the encoder and
// decoder perceptrons of eqs. (i) and (iii), forward and backward, and the
// masked mean squared error on the interior points.  Everything is float32
// with sums in a fixed order (block partials reduced in block order), so the
// results are bitwise reproducible.
#include <algorithm>

#include "common.hpp"

using namespace dsmp;

namespace {

constexpr int ROWS_PER_PART = 256;   // rows per partial of a weight-gradient sum

// out[n][o] = act(b[o] + sum_i in[n][i] W[o][i]), the sum as a chain of fused
// multiply-adds in input order; optional bf16 copy of the output.
__global__ __launch_bounds__(256) void k_dense(int64_t n, int din, int dout, const float* __restrict__ in,
                                               const float* __restrict__ W, const float* __restrict__ b, int relu,
                                               float* __restrict__ out, __bf16* __restrict__ out_bf16) {
  const int64_t total = n * dout;
  for (int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x; x < total; x += (int64_t)gridDim.x * 256) {
    const int64_t r = x / dout;
    const int o = (int)(x % dout);
    const float* xi = in + r * din;
    const float* wo = W + (int64_t)o * din;
    float v = b[o];
#pragma unroll 8
    for (int i = 0; i < din; ++i) v = __builtin_fmaf(xi[i], wo[i], v);
    if (relu && !(v > 0.0f)) v = 0.0f;
    out[x] = v;
    if (out_bf16) out_bf16[x] = (__bf16)v;
  }
}

// gin[n][i] (+)= [h[n][i] > 0] * sum_o g[n][o] W[o][i]   (mask h optional)
__global__ __launch_bounds__(256) void k_dense_back(int64_t n, int din, int dout, const float* __restrict__ g,
                                                    const float* __restrict__ W, const float* __restrict__ h,
                                                    float* __restrict__ gin, int accumulate) {
  const int64_t total = n * din;
  for (int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x; x < total; x += (int64_t)gridDim.x * 256) {
    const int64_t r = x / din;
    const int i = (int)(x % din);
    const float* gr = g + r * dout;
    float v = 0.0f;
#pragma unroll 8
    for (int o = 0; o < dout; ++o) v = __builtin_fmaf(gr[o], W[(int64_t)o * din + i], v);
    if (h && !(h[x] > 0.0f)) v = 0.0f;
    gin[x] = accumulate ? gin[x] + v : v;
  }
}

// part[c][o][i] = sum over rows r of part c of g[r][o] * in[r][i] for i < din,
// and part[c][o][din] = sum of g[r][o] (the bias gradient, against a column of
// ones), rows in order.  Block (c, b) serves the 256 (o, i) pairs starting at
// 256 b; the rows pass through LDS 32 at a time.
constexpr int OUTER_RC = 32;

__global__ __launch_bounds__(256) void k_outer_rows(int64_t n, int din, int dout, const float* __restrict__ g,
                                                    const float* __restrict__ in, float* __restrict__ part) {
  __shared__ float gs[OUTER_RC * 256], xs[OUTER_RC * 257];
  const int64_t r0 = (int64_t)blockIdx.x * ROWS_PER_PART;
  const int64_t r1 = std::min<int64_t>(r0 + ROWS_PER_PART, n);
  const int pairs = dout * (din + 1), xw = din + 1;
  const int p = blockIdx.y * 256 + threadIdx.x;
  const int o = p / xw, i = p % xw;
  float v = 0.0f;
  for (int64_t rc = r0; rc < r1; rc += OUTER_RC) {
    const int cnt = (int)std::min<int64_t>(OUTER_RC, r1 - rc);
    __syncthreads();
    for (int t = threadIdx.x; t < cnt * dout; t += 256) gs[t] = g[rc * dout + t];
    for (int t = threadIdx.x; t < cnt * xw; t += 256) {
      const int k = t / xw, c = t % xw;
      xs[t] = c < din ? in[(rc + k) * din + c] : 1.0f;
    }
    __syncthreads();
    if (p < pairs)
      for (int k = 0; k < cnt; ++k) v = __builtin_fmaf(gs[k * dout + o], xs[k * xw + i], v);
  }
  if (p < pairs) part[(int64_t)blockIdx.x * pairs + p] = v;
}

dim3 outer_grid(int np, int din, int dout) { return dim3(np, ceil_div(dout * (din + 1), 256)); }

// dW[o][i] (+)= sum_c part[c][o][i], db[o] (+)= sum_c part[c][o][din], for
// the three weight gradients of a perceptron in one launch: segment m takes
// the blocks [first[m], first[m + 1]).  A block serves 64 pairs; its four
// waves sum the partials c = g, g+4, ... in order and the four sums are
// added in wave order (a fixed order).
struct OuterFinal3 {
  const float* part[3];
  float* dW[3];
  float* db[3];
  int din[3], dout[3], first[4];
  int nparts, accumulate;
};


__global__ __launch_bounds__(256) void k_outer_final3(OuterFinal3 a) {
  __shared__ float sh[4][64];
  const int m = (int)blockIdx.x < a.first[1] ? 0 : (int)blockIdx.x < a.first[2] ? 1 : 2;
  const int din = a.din[m], dout = a.dout[m], nparts = a.nparts;
  const float* part = a.part[m];
  const int pairs = dout * (din + 1);
  const int p = ((int)blockIdx.x - a.first[m]) * 64 + (threadIdx.x & 63), g = threadIdx.x >> 6;
  float v = 0.0f;
  if (p < pairs) {
#pragma unroll 8
    for (int c = g; c < nparts; c += 4) v += part[(int64_t)c * pairs + p];
  }
  sh[g][threadIdx.x & 63] = v;
  __syncthreads();
  if (g == 0 && p < pairs) {
    v = sh[0][threadIdx.x] + sh[1][threadIdx.x] + sh[2][threadIdx.x] + sh[3][threadIdx.x];
    const int o = p / (din + 1), i = p % (din + 1);
    float* t = i < din ? a.dW[m] + (int64_t)o * din + i : a.db[m] + o;
    *t = a.accumulate ? *t + v : v;
  }
}

// Fused perceptron passes over blocks of FR rows, activations in LDS (used
// when they fit, see fused_lds).  A dense step out[r][o] = act(b[o] +
// sum_k in[r][k] W[o][k]) over the block's rows, in LDS, with optional copies
// to global memory.
constexpr int FR = 32;

// WT: the layer's weights transposed, [K][O], in LDS.
__device__ __forceinline__ void dense_rows(int cnt, int K, int O, const float* __restrict__ in_s,
                                           const float* __restrict__ WT, const float* __restrict__ b, int relu,
                                           float* __restrict__ out_s, float* __restrict__ out_g,
                                           __bf16* __restrict__ out_bf16) {
  for (int t = threadIdx.x; t < cnt * O; t += 256) {
    const int r = t / O, o = t % O;
    const float* xi = in_s + r * K;
    float v = b[o];
#pragma unroll 8
    for (int k = 0; k < K; ++k) v = __builtin_fmaf(xi[k], WT[k * O + o], v);
    if (relu && !(v > 0.0f)) v = 0.0f;
    if (out_s) out_s[t] = v;
    if (out_g) out_g[t] = v;
    if (out_bf16) out_bf16[t] = (__bf16)v;
  }
}

// g_in[r][k] = [mask[r][k] > 0] * sum_o g[r][o] W[o][k] over the block's rows (in LDS)
__device__ __forceinline__ void dense_back_rows(int cnt, int K, int O, const float* __restrict__ g_s,
                                                const float* __restrict__ W, const float* __restrict__ mask_s,
                                                float* __restrict__ out_s, float* __restrict__ out_g, int accumulate) {
  for (int t = threadIdx.x; t < cnt * K; t += 256) {
    const int r = t / K, k = t % K;
    const float* gr = g_s + r * O;
    float v = 0.0f;
#pragma unroll 8
    for (int o = 0; o < O; ++o) v = __builtin_fmaf(gr[o], W[(int64_t)o * K + k], v);
    if (mask_s && !(mask_s[t] > 0.0f)) v = 0.0f;
    if (out_s) out_s[t] = v;
    if (out_g) out_g[t] = accumulate ? out_g[t] + v : v;
  }
}

// part[o][k] = sum over the block's rows of g[r][o] * in[r][k] (k < K), part[o][K] = sum of g[r][o]
__device__ __forceinline__ void outer_block(int cnt, int K, int O, const float* __restrict__ g_s,
                                            const float* __restrict__ in_s, float* __restrict__ part) {
  for (int p = threadIdx.x; p < O * (K + 1); p += 256) {
    const int o = p / (K + 1), k = p % (K + 1);
    float v = 0.0f;
    if (k < K)
      for (int r = 0; r < cnt; ++r) v = __builtin_fmaf(g_s[r * O + o], in_s[r * K + k], v);
    else
      for (int r = 0; r < cnt; ++r) v += g_s[r * O + o];
    part[p] = v;
  }
}

struct MlpArgs {
  int64_t n;
  int din, dh, dout;
  const float *W1, *b1, *W2, *b2, *W3, *b3;
  const float* x;
  float *h1, *h2;        // saved activations [n][dh]
  float* y;              // forward output [n][dout]
  __bf16* y_bf16;
  const float* gy;       // backward input [n][dout]
  float* gx;             // backward output [n][din] (nullable)
  int gx_acc;
  float *p3, *p2, *p1;   // per-block partials of the weight gradients
};

// Persistent blocks: the three weight matrices are copied transposed into LDS
// once, then the blocks take FR-row tiles in turn.
__global__ __launch_bounds__(256) void k_mlp_fwd(MlpArgs a) {
  extern __shared__ float sm[];
  float* t1 = sm;                        // W1^T [din][dh]
  float* t2 = t1 + a.din * a.dh;         // W2^T [dh][dh]
  float* t3 = t2 + a.dh * a.dh;          // W3^T [dh][dout]
  float* xs = t3 + a.dh * a.dout;
  float* s1 = xs + FR * a.din;
  float* s2 = s1 + FR * a.dh;
  for (int t = threadIdx.x; t < a.din * a.dh; t += 256) t1[(t % a.din) * a.dh + t / a.din] = a.W1[t];
  for (int t = threadIdx.x; t < a.dh * a.dh; t += 256) t2[(t % a.dh) * a.dh + t / a.dh] = a.W2[t];
  for (int t = threadIdx.x; t < a.dout * a.dh; t += 256) t3[(t % a.dh) * a.dout + t / a.dh] = a.W3[t];
  const int64_t ntile = (a.n + FR - 1) / FR;
  for (int64_t tile = blockIdx.x; tile < ntile; tile += gridDim.x) {
    const int64_t r0 = tile * FR;
    const int cnt = (int)std::min<int64_t>(FR, a.n - r0);
    __syncthreads();   // weights staged / the previous tile's rows consumed
    for (int t = threadIdx.x; t < cnt * a.din; t += 256) xs[t] = a.x[r0 * a.din + t];
    __syncthreads();
    dense_rows(cnt, a.din, a.dh, xs, t1, a.b1, 1, s1, a.h1 + r0 * a.dh, nullptr);
    __syncthreads();
    dense_rows(cnt, a.dh, a.dh, s1, t2, a.b2, 1, s2, a.h2 + r0 * a.dh, nullptr);
    __syncthreads();
    dense_rows(cnt, a.dh, a.dout, s2, t3, a.b3, 0, nullptr, a.y + r0 * a.dout,
               a.y_bf16 ? a.y_bf16 + r0 * a.dout : nullptr);
  }
}

__global__ __launch_bounds__(256) void k_mlp_bwd(MlpArgs a) {
  extern __shared__ float sm[];
  float* xs = sm;                     // [FR][din]
  float* g3 = xs + FR * a.din;        // [FR][dout]
  float* s1 = g3 + FR * a.dout;       // h1 [FR][dh]
  float* s2 = s1 + FR * a.dh;         // h2
  float* g2 = s2 + FR * a.dh;
  float* g1 = g2 + FR * a.dh;
  const int64_t r0 = (int64_t)blockIdx.x * FR;
  const int cnt = (int)std::min<int64_t>(FR, a.n - r0);
  for (int t = threadIdx.x; t < cnt * a.din; t += 256) xs[t] = a.x[r0 * a.din + t];
  for (int t = threadIdx.x; t < cnt * a.dout; t += 256) g3[t] = a.gy[r0 * a.dout + t];
  for (int t = threadIdx.x; t < cnt * a.dh; t += 256) {
    s1[t] = a.h1[r0 * a.dh + t];
    s2[t] = a.h2[r0 * a.dh + t];
  }
  __syncthreads();
  dense_back_rows(cnt, a.dh, a.dout, g3, a.W3, s2, g2, nullptr, 0);
  __syncthreads();
  dense_back_rows(cnt, a.dh, a.dh, g2, a.W2, s1, g1, nullptr, 0);
  __syncthreads();
  if (a.gx) dense_back_rows(cnt, a.din, a.dh, g1, a.W1, nullptr, nullptr, a.gx + r0 * a.din, a.gx_acc);
  const int64_t b = blockIdx.x;
  outer_block(cnt, a.dh, a.dout, g3, s2, a.p3 + b * a.dout * (a.dh + 1));
  outer_block(cnt, a.dh, a.dh, g2, s1, a.p2 + b * a.dh * (a.dh + 1));
  outer_block(cnt, a.din, a.dh, g1, xs, a.p1 + b * a.dh * (a.din + 1));
}

// Matrix-core forms of the fused passes, for hidden widths that are whole
// 32-column tiles.  Every product is a chain of fp32 32x32x2 MFMA steps in
// contraction order (the accumulator starting from the bias, or zero), which
// rounds as the fused multiply-add chains above do.  Matrices sit in LDS in
// their natural row-major layout with one float of row padding, so both the
// row-indexed and the column-indexed operand reads are free of bank
// conflicts; rows of a tile past its end hold zeros.
typedef float f32x16m __attribute__((ext_vector_type(16)));

// C += sum over k < K of A(r, k) B(k, c) for the 32x32 block of rows
// [0, 32) and columns [c0, c0 + 32): A row-major with pitch pa, B given as
// Bt row-major [c][k] (pitch pb, rows >= nc read as zero), two k per step.
__device__ __forceinline__ f32x16m mchain_rows(f32x16m C, int K, const float* A, int pa, const float* Bt, int pb,
                                              int c0, int nc) {
  const int l = threadIdx.x & 63, r = l & 31, h = l >> 5;
  const bool cv = c0 + r < nc;
  for (int kk = 0; kk < K; kk += 2) {
    const int k = kk + h;
    const float av = k < K ? A[r * pa + k] : 0.0f;
    const float bv = k < K && cv ? Bt[(c0 + r) * pb + k] : 0.0f;
    C = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, C, 0, 0, 0);
  }
  return C;
}

// The same with B row-major [k][c] (pitch pb, columns >= nc read as zero).
__device__ __forceinline__ f32x16m mchain_cols(f32x16m C, int K, const float* A, int pa, const float* B, int pb,
                                              int c0, int nc) {
  const int l = threadIdx.x & 63, r = l & 31, h = l >> 5;
  const bool cv = c0 + r < nc;
  for (int kk = 0; kk < K; kk += 2) {
    const int k = kk + h;
    const float av = k < K ? A[r * pa + k] : 0.0f;
    const float bv = k < K && cv ? B[k * pb + c0 + r] : 0.0f;
    C = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, C, 0, 0, 0);
  }
  return C;
}

// out[r][o] = act(b[o] + sum_k in[r][k] W[o][k]) for the tile's rows, one
// 32-column block per wave in turn; to LDS (pitch O + 1) and global memory.
__device__ __forceinline__ void mdense(int cnt, int K, int O, const float* in_s, const float* W_s, const float* b,
                                       int relu, float* out_s, float* out_g, __bf16* out_bf16) {
  const int l = threadIdx.x & 63, wv = threadIdx.x >> 6, r = l & 31, h = l >> 5;
  for (int ob = wv; ob * 32 < O; ob += 4) {
    const int c = ob * 32 + r;
    const float bc = c < O ? b[c] : 0.0f;
    f32x16m C;
#pragma unroll
    for (int i = 0; i < 16; ++i) C[i] = bc;
    C = mchain_rows(C, K, in_s, K + 1, W_s, K + 1, ob * 32, O);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = 8 * (i / 4) + 4 * h + (i % 4);
      float v = C[i];
      if (relu && !(v > 0.0f)) v = 0.0f;
      if (c < O) {
        if (out_s) out_s[row * (O + 1) + c] = row < cnt ? v : 0.0f;
        if (row < cnt) {
          if (out_g) out_g[(int64_t)row * O + c] = v;
          if (out_bf16) out_bf16[(int64_t)row * O + c] = (__bf16)v;
        }
      }
    }
  }
}

// gin[r][k] = [mask[r][k] > 0] * sum_o g[r][o] W[o][k]: A = g (pitch O + 1),
// B = W row-major [o][k] (pitch K + 1); to LDS (pitch K + 1) and/or global.
__device__ __forceinline__ void mdense_back(int cnt, int K, int O, const float* g_s, const float* W_s,
                                            const float* mask_s, float* out_s, float* out_g, int accumulate) {
  const int l = threadIdx.x & 63, wv = threadIdx.x >> 6, r = l & 31, h = l >> 5;
  for (int kb = wv; kb * 32 < K; kb += 4) {
    const int c = kb * 32 + r;
    f32x16m C = f32x16m{};
    C = mchain_cols(C, O, g_s, O + 1, W_s, K + 1, kb * 32, K);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = 8 * (i / 4) + 4 * h + (i % 4);
      if (c >= K) continue;
      float v = C[i];
      if (mask_s && !(mask_s[row * (K + 1) + c] > 0.0f)) v = 0.0f;
      if (out_s) out_s[row * (K + 1) + c] = row < cnt ? v : 0.0f;
      if (out_g && row < cnt) {
        float* t = out_g + (int64_t)row * K + c;
        *t = accumulate ? *t + v : v;
      }
    }
  }
}

// part[o][k] = sum over the tile's rows r of g[r][o] in[r][k] (k < K) and
// part[o][K] = sum of g[r][o]: rows of the product are o (A = g transposed,
// read as g[r][o]), its contraction index the tile's rows.
__device__ __forceinline__ void mouter(int K, int O, const float* g_s, const float* in_s, float* part) {
  const int l = threadIdx.x & 63, wv = threadIdx.x >> 6, r = l & 31, h = l >> 5;
  const int nob = (O + 31) / 32, nkb = (K + 1 + 31) / 32;
  for (int t = wv; t < nob * nkb; t += 4) {
    const int ob = t / nkb, kb = t % nkb;
    const int o = ob * 32 + r, c = kb * 32 + r;
    f32x16m C = f32x16m{};
    for (int kk = 0; kk < FR; kk += 2) {
      const int rr = kk + h;
      const float av = o < O ? g_s[rr * (O + 1) + o] : 0.0f;
      const float bv = c < K ? in_s[rr * (K + 1) + c] : (c == K ? 1.0f : 0.0f);
      C = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, C, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int oo = ob * 32 + 8 * (i / 4) + 4 * h + (i % 4);
      if (oo < O && c <= K) part[oo * (K + 1) + c] = C[i];
    }
  }
}

// A [rows][w] row-major global matrix (w <= 256) to LDS with pitch w + 1,
// rows past `valid` as zeros: each thread keeps one column and steps over
// the rows 256 / w at a time (one division per thread, none per element).
__device__ __forceinline__ void stage_mat(float* dst, const float* src, int rows, int w, int valid) {
  const int per = 256 / w, t = threadIdx.x, r0 = t / w, c = t - r0 * w;
  if (r0 >= per) return;
  for (int rr = r0; rr < rows; rr += per)
    dst[rr * (w + 1) + c] = rr < valid ? src[(int64_t)rr * w + c] : 0.0f;
}

// Rows [0, cnt) of a [*][w] global matrix to LDS with pitch w + 1, zeros past cnt.
__device__ __forceinline__ void stage_rows(float* dst, const float* src, int cnt, int w) {
  stage_mat(dst, src, FR, w, cnt);
}

struct MlpLdsM {
  int w1, w2, w3, x, s1, s2, g3, g2, g1, fwd, bwd;   // float offsets / totals
};

__host__ __device__ inline MlpLdsM mlp_lds_m(int din, int dh, int dout) {
  MlpLdsM m;
  m.w1 = 0;
  m.w2 = m.w1 + dh * (din + 1);
  m.w3 = m.w2 + dh * (dh + 1);
  m.x = m.w3 + dout * (dh + 1);
  m.s1 = m.x + FR * (din + 1);
  m.s2 = m.s1 + FR * (dh + 1);
  m.fwd = m.s2 + FR * (dh + 1);
  m.g3 = m.fwd;
  m.g2 = m.g3 + FR * (dout + 1);
  m.g1 = m.g2 + FR * (dh + 1);
  m.bwd = m.g1 + FR * (dh + 1);
  return m;
}

__global__ __launch_bounds__(256) void k_mlp_fwd_m(MlpArgs a) {
  extern __shared__ float sm[];
  const MlpLdsM m = mlp_lds_m(a.din, a.dh, a.dout);
  stage_mat(sm + m.w1, a.W1, a.dh, a.din, a.dh);
  stage_mat(sm + m.w2, a.W2, a.dh, a.dh, a.dh);
  stage_mat(sm + m.w3, a.W3, a.dout, a.dh, a.dout);
  const int64_t ntile = (a.n + FR - 1) / FR;
  for (int64_t tile = blockIdx.x; tile < ntile; tile += gridDim.x) {
    const int64_t r0 = tile * FR;
    const int cnt = (int)std::min<int64_t>(FR, a.n - r0);
    __syncthreads();   // weights staged / the previous tile consumed
    stage_rows(sm + m.x, a.x + r0 * a.din, cnt, a.din);
    __syncthreads();
    mdense(cnt, a.din, a.dh, sm + m.x, sm + m.w1, a.b1, 1, sm + m.s1, a.h1 + r0 * a.dh, nullptr);
    __syncthreads();
    mdense(cnt, a.dh, a.dh, sm + m.s1, sm + m.w2, a.b2, 1, sm + m.s2, a.h2 + r0 * a.dh, nullptr);
    __syncthreads();
    mdense(cnt, a.dh, a.dout, sm + m.s2, sm + m.w3, a.b3, 0, nullptr, a.y + r0 * a.dout,
           a.y_bf16 ? a.y_bf16 + r0 * a.dout : nullptr);
  }
}

__global__ __launch_bounds__(256) void k_mlp_bwd_m(MlpArgs a) {
  extern __shared__ float sm[];
  const MlpLdsM m = mlp_lds_m(a.din, a.dh, a.dout);
  const int64_t r0 = (int64_t)blockIdx.x * FR;
  const int cnt = (int)std::min<int64_t>(FR, a.n - r0);
  stage_mat(sm + m.w1, a.W1, a.dh, a.din, a.dh);
  stage_mat(sm + m.w2, a.W2, a.dh, a.dh, a.dh);
  stage_mat(sm + m.w3, a.W3, a.dout, a.dh, a.dout);
  stage_rows(sm + m.x, a.x + r0 * a.din, cnt, a.din);
  stage_rows(sm + m.g3, a.gy + r0 * a.dout, cnt, a.dout);
  stage_rows(sm + m.s1, a.h1 + r0 * a.dh, cnt, a.dh);
  stage_rows(sm + m.s2, a.h2 + r0 * a.dh, cnt, a.dh);
  __syncthreads();
  mdense_back(cnt, a.dh, a.dout, sm + m.g3, sm + m.w3, sm + m.s2, sm + m.g2, nullptr, 0);
  __syncthreads();
  mdense_back(cnt, a.dh, a.dh, sm + m.g2, sm + m.w2, sm + m.s1, sm + m.g1, nullptr, 0);
  __syncthreads();
  if (a.gx) mdense_back(cnt, a.din, a.dh, sm + m.g1, sm + m.w1, nullptr, nullptr, a.gx + r0 * a.din, a.gx_acc);
  const int64_t b = blockIdx.x;
  mouter(a.dh, a.dout, sm + m.g3, sm + m.s2, a.p3 + b * a.dout * (a.dh + 1));
  mouter(a.dh, a.dh, sm + m.g2, sm + m.s1, a.p2 + b * a.dh * (a.dh + 1));
  mouter(a.din, a.dh, sm + m.g1, sm + m.x, a.p1 + b * a.dh * (a.din + 1));
}

// LDS bytes of the matrix-core passes (at most 96 KB: two workgroups per
// CU); 0 when they do not apply
int mfma_lds(const dsmp_mlp_desc& d) {
  if (d.d_hid % 32 != 0) return 0;
  const MlpLdsM m = mlp_lds_m(d.d_in, d.d_hid, d.d_out);
  const size_t bytes = (size_t)std::max(m.fwd, m.bwd) * sizeof(float);
  return bytes <= 96 * 1024 ? (int)bytes : 0;
}

dsmp_status allow_lds(dsmp_handle* h, const void* kern, int bytes) {
  DSMP_HIP(h, hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, bytes));
  return DSMP_OK;
}

// LDS bytes of the fused passes; 0 when either does not fit (64 KB)
int fused_fwd_lds(const dsmp_mlp_desc& d) {
  return (int)(((size_t)d.d_in * d.d_hid + (size_t)d.d_hid * d.d_hid + (size_t)d.d_hid * d.d_out +
                (size_t)FR * (d.d_in + 2 * d.d_hid)) * sizeof(float));
}
int fused_lds(const dsmp_mlp_desc& d) {
  const size_t bytes = (size_t)FR * (d.d_in + d.d_out + 4 * d.d_hid) * sizeof(float);
  return bytes <= 64 * 1024 && fused_fwd_lds(d) <= 64 * 1024 ? (int)bytes : 0;
}

// Masked MSE: per-block partial sums (squared error, interior rows), a
// single-block final sum, then the gradient.
__global__ __launch_bounds__(256) void k_mse_partial(int64_t n, int c, const float* __restrict__ pred,
                                                     const float* __restrict__ target,
                                                     const uint8_t* __restrict__ mask, float2* __restrict__ part) {
  __shared__ float ss[256], sk[256];
  const int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
  float s = 0.0f, k = 0.0f;
  if (r < n && mask[r]) {
    for (int j = 0; j < c; ++j) {
      const float dlt = pred[r * c + j] - target[r * c + j];
      s = __builtin_fmaf(dlt, dlt, s);
    }
    k = 1.0f;
  }
  ss[threadIdx.x] = s;
  sk[threadIdx.x] = k;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) {
      ss[threadIdx.x] += ss[threadIdx.x + w];
      sk[threadIdx.x] += sk[threadIdx.x + w];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) part[blockIdx.x] = make_float2(ss[0], sk[0]);
}

__global__ __launch_bounds__(256) void k_mse_final(int nparts, int c, const float2* __restrict__ part,
                                                   float* __restrict__ loss, float* __restrict__ scale) {
  __shared__ double ss[256], sk[256];
  double s = 0.0, k = 0.0;
  for (int p = threadIdx.x; p < nparts; p += 256) {
    s += part[p].x;
    k += part[p].y;
  }
  ss[threadIdx.x] = s;
  sk[threadIdx.x] = k;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) {
      ss[threadIdx.x] += ss[threadIdx.x + w];
      sk[threadIdx.x] += sk[threadIdx.x + w];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double cnt = sk[0] * c;
    *loss = cnt > 0 ? (float)(ss[0] / cnt) : 0.0f;
    *scale = cnt > 0 ? (float)(2.0 / cnt) : 0.0f;
  }
}

__global__ __launch_bounds__(256) void k_mse_grad(int64_t n, int c, const float* __restrict__ pred,
                                                  const float* __restrict__ target, const uint8_t* __restrict__ mask,
                                                  const float* __restrict__ scale, float* __restrict__ grad) {
  const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (x >= n * c) return;
  grad[x] = mask[x / c] ? (pred[x] - target[x]) * *scale : 0.0f;
}

struct MlpSaved {
  float *h1, *h2;
  size_t total;
};

MlpSaved mlp_saved(const dsmp_mlp_desc& d, int64_t n, void* base) {
  Carve c(base);
  MlpSaved s;
  s.h1 = c.take<float>((size_t)n * d.d_hid);
  s.h2 = c.take<float>((size_t)n * d.d_hid);
  s.total = c.used();
  return s;
}

struct MlpWs {
  float *g2, *g1, *p3, *p2, *p1;
  int nparts;
  size_t total;
};

MlpWs mlp_ws(const dsmp_mlp_desc& d, int64_t n, void* base) {
  Carve c(base);
  MlpWs w;
  w.nparts = (int)std::max<int64_t>(1, ceil_div(n, (mfma_lds(d) || fused_lds(d)) ? FR : ROWS_PER_PART));
  w.g2 = c.take<float>((size_t)n * d.d_hid);
  w.g1 = c.take<float>((size_t)n * d.d_hid);
  w.p3 = c.take<float>((size_t)w.nparts * d.d_out * (d.d_hid + 1));
  w.p2 = c.take<float>((size_t)w.nparts * d.d_hid * (d.d_hid + 1));
  w.p1 = c.take<float>((size_t)w.nparts * d.d_hid * (d.d_in + 1));
  w.total = c.used();
  return w;
}

dsmp_status check_mlp(dsmp_handle* h, const dsmp_mlp_desc* d) {
  DSMP_CHECK(h, d, DSMP_INVALID_ARG, "desc is NULL");
  DSMP_CHECK(h, d->d_in >= 1 && d->d_in <= 256 && d->d_out >= 1 && d->d_out <= 256 && d->d_hid >= 4 &&
                    d->d_hid <= 256 && d->d_hid % 4 == 0,
             DSMP_UNSUPPORTED, "unsupported perceptron widths %d -> %d -> %d", d->d_in, d->d_hid, d->d_out);
  return DSMP_OK;
}

unsigned grid_for(int64_t total) { return (unsigned)std::min<int64_t>(ceil_div(total, 256), 65536); }

}  // namespace

extern "C" dsmp_status dsmp_mlp_workspace(const dsmp_mlp_desc* desc, int64_t n, size_t* saved_bytes,
                                          size_t* bwd_ws_bytes) {
  if (!desc || !saved_bytes || !bwd_ws_bytes || n < 0) return DSMP_INVALID_ARG;
  if (check_mlp(nullptr, desc) != DSMP_OK) return DSMP_UNSUPPORTED;
  *saved_bytes = mlp_saved(*desc, n, nullptr).total;
  *bwd_ws_bytes = mlp_ws(*desc, n, nullptr).total;
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_mlp_forward(dsmp_handle* h, const dsmp_mlp_desc* desc, const dsmp_mlp_params* p,
                                        const float* x, int64_t n, float* y, void* y_bf16, void* saved,
                                        size_t saved_bytes) {
  if (!h) return DSMP_INVALID_ARG;
  dsmp_status st = check_mlp(h, desc);
  if (st != DSMP_OK) return st;
  const dsmp_mlp_desc& d = *desc;
  DSMP_CHECK(h, n >= 0 && n < (int64_t)1 << 31, DSMP_INVALID_ARG, "row count out of range");
  DSMP_CHECK(h, p && p->W1 && p->b1 && p->W2 && p->b2 && p->W3 && p->b3, DSMP_INVALID_ARG, "a parameter is NULL");
  DSMP_CHECK(h, n == 0 || (x && y && saved), DSMP_INVALID_ARG, "a data pointer is NULL");
  const MlpSaved s = mlp_saved(d, n, saved);
  DSMP_CHECK(h, saved_bytes >= s.total, DSMP_WORKSPACE_TOO_SMALL, "saved buffer needs %zu bytes", s.total);
  if (n == 0) return DSMP_OK;
  ProfScope prof(h, DSMP_K_MLP);
  hipStream_t st_ = h->stream;
  if (const int lds = mfma_lds(d)) {
    MlpArgs a{n, d.d_in, d.d_hid, d.d_out, p->W1, p->b1, p->W2, p->b2, p->W3, p->b3, x, s.h1, s.h2, y,
              static_cast<__bf16*>(y_bf16), nullptr, nullptr, 0, nullptr, nullptr, nullptr};
    const int64_t grid = std::min<int64_t>(ceil_div(n, FR), (int64_t)h->n_cu * 2);
    if ((st = allow_lds(h, reinterpret_cast<const void*>(k_mlp_fwd_m), lds)) != DSMP_OK) return st;
    hipLaunchKernelGGL(k_mlp_fwd_m, dim3((unsigned)grid), dim3(256), lds, st_, a);
    DSMP_LAUNCHED(h, "perceptron forward");
    return DSMP_OK;
  }
  if (const int lds = fused_lds(d)) {
    MlpArgs a{n, d.d_in, d.d_hid, d.d_out, p->W1, p->b1, p->W2, p->b2, p->W3, p->b3, x, s.h1, s.h2, y,
              static_cast<__bf16*>(y_bf16), nullptr, nullptr, 0, nullptr, nullptr, nullptr};
    (void)lds;
    const int64_t grid = std::min<int64_t>(ceil_div(n, FR), (int64_t)h->n_cu * 2);
    hipLaunchKernelGGL(k_mlp_fwd, dim3((unsigned)grid), dim3(256), fused_fwd_lds(d), st_, a);
    DSMP_LAUNCHED(h, "perceptron forward");
    return DSMP_OK;
  }
  hipLaunchKernelGGL(k_dense, dim3(grid_for(n * d.d_hid)), dim3(256), 0, st_, n, d.d_in, d.d_hid, x, p->W1, p->b1, 1,
                     s.h1, (__bf16*)nullptr);
  hipLaunchKernelGGL(k_dense, dim3(grid_for(n * d.d_hid)), dim3(256), 0, st_, n, d.d_hid, d.d_hid, s.h1, p->W2, p->b2,
                     1, s.h2, (__bf16*)nullptr);
  hipLaunchKernelGGL(k_dense, dim3(grid_for(n * d.d_out)), dim3(256), 0, st_, n, d.d_hid, d.d_out, s.h2, p->W3, p->b3,
                     0, y, static_cast<__bf16*>(y_bf16));
  DSMP_LAUNCHED(h, "perceptron forward");
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_mlp_backward(dsmp_handle* h, const dsmp_mlp_desc* desc, const dsmp_mlp_params* p,
                                         const float* x, int64_t n, const void* saved, size_t saved_bytes,
                                         const float* grad_y, float* grad_x, const dsmp_mlp_grads* grads,
                                         int32_t flags, void* ws, size_t ws_bytes) {
  if (!h) return DSMP_INVALID_ARG;
  dsmp_status st = check_mlp(h, desc);
  if (st != DSMP_OK) return st;
  const dsmp_mlp_desc& d = *desc;
  DSMP_CHECK(h, n >= 0 && n < (int64_t)1 << 31, DSMP_INVALID_ARG, "row count out of range");
  DSMP_CHECK(h, p && p->W1 && p->b1 && p->W2 && p->b2 && p->W3 && p->b3, DSMP_INVALID_ARG, "a parameter is NULL");
  DSMP_CHECK(h, grads && grads->dW1 && grads->db1 && grads->dW2 && grads->db2 && grads->dW3 && grads->db3,
             DSMP_INVALID_ARG, "a gradient pointer is NULL");
  DSMP_CHECK(h, n == 0 || (x && saved && grad_y), DSMP_INVALID_ARG, "a data pointer is NULL");
  DSMP_CHECK(h, (flags & ~(DSMP_GRAD_ACCUMULATE | DSMP_GRAD_X_ACCUMULATE)) == 0, DSMP_INVALID_ARG, "unknown flags");
  const MlpSaved s = mlp_saved(d, n, const_cast<void*>(saved));
  DSMP_CHECK(h, saved_bytes >= s.total, DSMP_WORKSPACE_TOO_SMALL, "saved buffer needs %zu bytes", s.total);
  const MlpWs need = mlp_ws(d, n, nullptr);
  DSMP_CHECK(h, ws && ws_bytes >= need.total, DSMP_WORKSPACE_TOO_SMALL, "backward workspace needs %zu bytes",
             need.total);
  const MlpWs w = mlp_ws(d, n, ws);
  const int acc = flags & DSMP_GRAD_ACCUMULATE;
  ProfScope prof(h, DSMP_K_MLP);
  hipStream_t q = h->stream;
  const int np = n > 0 ? w.nparts : 0;
  if (n > 0 && mfma_lds(d)) {
    MlpArgs a{n, d.d_in, d.d_hid, d.d_out, p->W1, p->b1, p->W2, p->b2, p->W3, p->b3, x, s.h1, s.h2, nullptr,
              nullptr, grad_y, grad_x, (flags & DSMP_GRAD_X_ACCUMULATE) ? 1 : 0, w.p3, w.p2, w.p1};
    if ((st = allow_lds(h, reinterpret_cast<const void*>(k_mlp_bwd_m), mfma_lds(d))) != DSMP_OK) return st;
    hipLaunchKernelGGL(k_mlp_bwd_m, dim3(np), dim3(256), mfma_lds(d), q, a);
  } else if (n > 0 && fused_lds(d)) {
    MlpArgs a{n, d.d_in, d.d_hid, d.d_out, p->W1, p->b1, p->W2, p->b2, p->W3, p->b3, x, s.h1, s.h2, nullptr,
              nullptr, grad_y, grad_x, (flags & DSMP_GRAD_X_ACCUMULATE) ? 1 : 0, w.p3, w.p2, w.p1};
    hipLaunchKernelGGL(k_mlp_bwd, dim3(np), dim3(256), fused_lds(d), q, a);
  } else if (n > 0) {
    // layer 3 (no activation): weights from grad_y and h2, then back to h2's pre-activation
    hipLaunchKernelGGL(k_outer_rows, outer_grid(np, d.d_hid, d.d_out), dim3(256), 0, q, n, d.d_hid, d.d_out, grad_y,
                       s.h2, w.p3);
    hipLaunchKernelGGL(k_dense_back, dim3(grid_for(n * d.d_hid)), dim3(256), 0, q, n, d.d_hid, d.d_out, grad_y, p->W3,
                       s.h2, w.g2, 0);
    hipLaunchKernelGGL(k_outer_rows, outer_grid(np, d.d_hid, d.d_hid), dim3(256), 0, q, n, d.d_hid, d.d_hid, w.g2,
                       s.h1, w.p2);
    hipLaunchKernelGGL(k_dense_back, dim3(grid_for(n * d.d_hid)), dim3(256), 0, q, n, d.d_hid, d.d_hid, w.g2, p->W2,
                       s.h1, w.g1, 0);
    hipLaunchKernelGGL(k_outer_rows, outer_grid(np, d.d_in, d.d_hid), dim3(256), 0, q, n, d.d_in, d.d_hid, w.g1, x,
                       w.p1);
    if (grad_x)
      hipLaunchKernelGGL(k_dense_back, dim3(grid_for(n * d.d_in)), dim3(256), 0, q, n, d.d_in, d.d_hid, w.g1, p->W1,
                         (const float*)nullptr, grad_x, (flags & DSMP_GRAD_X_ACCUMULATE) ? 1 : 0);
  }
  // with no rows the partial count is 0 and the finals write zeros (or add nothing)
  OuterFinal3 f{{w.p3, w.p2, w.p1}, {grads->dW3, grads->dW2, grads->dW1}, {grads->db3, grads->db2, grads->db1},
                {d.d_hid, d.d_hid, d.d_in}, {d.d_out, d.d_hid, d.d_hid}, {0, 0, 0, 0}, np, acc};
  for (int m = 0; m < 3; ++m) f.first[m + 1] = f.first[m] + (int)ceil_div(f.dout[m] * (f.din[m] + 1), 64);
  hipLaunchKernelGGL(k_outer_final3, dim3((unsigned)f.first[3]), dim3(256), 0, q, f);
  DSMP_LAUNCHED(h, "perceptron backward");
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_masked_mse_workspace(int64_t n, size_t* bytes) {
  if (!bytes || n < 0) return DSMP_INVALID_ARG;
  Carve c(nullptr);
  c.take<float2>((size_t)std::max<int64_t>(1, ceil_div(n, 256)));
  c.take<float>(1);
  *bytes = c.used();
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_masked_mse(dsmp_handle* h, const float* pred, const float* target, const uint8_t* mask,
                                       int64_t n, int32_t c, float* loss, float* grad, void* ws, size_t ws_bytes) {
  if (!h) return DSMP_INVALID_ARG;
  DSMP_CHECK(h, n >= 0 && n < (int64_t)1 << 31 && c >= 1 && c <= 1024, DSMP_INVALID_ARG, "sizes out of range");
  DSMP_CHECK(h, loss && (n == 0 || (pred && target && mask)), DSMP_INVALID_ARG, "a pointer is NULL");
  size_t need = 0;
  dsmp_masked_mse_workspace(n, &need);
  DSMP_CHECK(h, ws && ws_bytes >= need, DSMP_WORKSPACE_TOO_SMALL, "workspace needs %zu bytes", need);
  Carve cv(ws);
  const int nparts = (int)(n > 0 ? ceil_div(n, 256) : 0);
  float2* part = cv.take<float2>((size_t)std::max(nparts, 1));
  float* scale = cv.take<float>(1);
  ProfScope prof(h, DSMP_K_LOSS);
  if (nparts > 0)
    hipLaunchKernelGGL(k_mse_partial, dim3(nparts), dim3(256), 0, h->stream, n, (int)c, pred, target, mask, part);
  hipLaunchKernelGGL(k_mse_final, dim3(1), dim3(256), 0, h->stream, nparts, (int)c, part, loss, scale);
  if (grad && n > 0)
    hipLaunchKernelGGL(k_mse_grad, dim3(ceil_div(n * c, 256)), dim3(256), 0, h->stream, n, (int)c, pred, target,
                       mask, scale, grad);
  DSMP_LAUNCHED(h, "masked mean squared error");
  return DSMP_OK;
}
