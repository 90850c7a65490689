// NNConv layer internals: MFMA fragment traits, packed parameter layout and
// the shapes each kernel instantiation is compiled for.
#pragma once

#include "common.hpp"

namespace dsmp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// One 32x32 output tile per MFMA chain.  Operand layouts (lane l, h = l/32):
//   A[row = l%32][k = ks*KS + h*EPL + t]   B[k = ks*KS + h*EPL + t][col = l%32]
//   D[row = 8*(i/4) + 4*h + (i%4)][col = l%32]  for accumulator register i.
template <typename T>
struct MT;

template <>
struct MT<__bf16> {
  static constexpr int KS = 16, EPL = 8;
  typedef bf16x8 frag;
  static __device__ __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

template <>
struct MT<float> {
  static constexpr int KS = 2, EPL = 1;
  typedef float frag;
  static __device__ __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

// Eight floats to one bf16x8 fragment with four packed conversions
// (round to nearest even), or one float to an fp32 fragment.
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

template <typename T>
__device__ __forceinline__ typename MT<T>::frag pack_frag(const float* v);

template <>
__device__ __forceinline__ bf16x8 pack_frag<__bf16>(const float* v) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bf16x2 b = __builtin_convertvector((f32x2){v[2 * i], v[2 * i + 1]}, bf16x2);
    w[i] = __builtin_bit_cast(uint32_t, b);
  }
  const uint4 u = make_uint4(w[0], w[1], w[2], w[3]);
  return __builtin_bit_cast(bf16x8, u);
}

template <>
__device__ __forceinline__ float pack_frag<float>(const float* v) { return v[0]; }

// A contraction index that comes out of a D tile (rows of the previous
// product) is consumed as the B operand of the next product straight from
// registers.  Register order n = 16*c + i of 32-row tile c maps to B element
// (ks = n / EPL, t = n % EPL); the weights on the A side are stored with
// their columns permuted to match:  packed column kk = ks*KS + h*EPL + t
// holds original column  k = 32*c + 8*(i/4) + 4*h + (i%4).
template <typename T>
__host__ __device__ __forceinline__ int kperm(int kk) {
  constexpr int KS = MT<T>::KS, EPL = MT<T>::EPL;
  int ks = kk / KS, rem = kk % KS, h = rem / EPL, t = rem % EPL;
  int n = ks * EPL + t, c = n / 16, i = n % 16;
  return 32 * c + 8 * (i / 4) + 4 * h + (i % 4);
}

// Direct global-to-LDS staging of a weight block (no registers on the way):
// ROWS rows of RB bytes, contiguous in global memory, land in LDS with a row
// pitch of RB + 16 bytes, which keeps the 32-row fragment reads free of bank
// conflicts.  Each wave-wide load fills 64 consecutive 16-byte LDS units; a
// unit in a row's padding slot re-reads that row's first unit, and lanes past
// the end of the block are masked off.  The copy is complete for the whole
// workgroup after stage_wait() and a barrier.
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void gbl_void_t;

template <int ROWS, int RB>
struct LdsStage {
  static constexpr int NU = RB / 16, PITCH = NU + 1, UNITS = ROWS * PITCH;
  static constexpr int PER = (UNITS + 255) / 256;
  static constexpr int BYTES = ROWS * (RB + 16);
  static_assert(RB % 16 == 0, "rows are whole 16-byte units");
  uint32_t off[PER];

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int U = i * 256 + (int)threadIdx.x;
      const int r = U / PITCH, u = U % PITCH;
      off[i] = (uint32_t)(r * RB + (u < NU ? u : 0) * 16);
    }
  }
  // Start the copy of the block at src into dst (ROWS * (RB + 16) bytes).
  __device__ __forceinline__ void issue(const unsigned char* src, unsigned char* dst) const {
    const int wbase = (int)(threadIdx.x & ~63u);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      if (UNITS % 256 == 0 || i + 1 < PER || i * 256 + (int)threadIdx.x < UNITS) {
        // keep the offset a 32-bit register at the load (scalar base + vector offset)
        uint32_t o = off[i];
        asm volatile("" : "+v"(o));
        __builtin_amdgcn_global_load_lds((gbl_void_t*)(src + o),
                                         (lds_void_t*)(dst + (size_t)(i * 256 + wbase) * 16), 16, 0, 0);
      }
    }
  }
};

// Cache policy of a global-to-LDS copy: the non-temporal (streaming) hint, for
// whole-kilobyte pieces of data read once and far larger than the caches.
constexpr int LDS_COPY_STREAM = 2;

// Copy n16 contiguous 16-byte units from global memory to contiguous LDS
// (each wave-wide load one contiguous kilobyte).
template <int POLICY = 0>
__device__ __forceinline__ void lds_copy_async(const unsigned char* src, unsigned char* dst, int n16) {
  const int tid = (int)threadIdx.x, wbase = tid & ~63;
  for (int i = 0; i * 256 < n16; ++i) {
    const int U = i * 256 + tid;
    if (U < n16)
      __builtin_amdgcn_global_load_lds((gbl_void_t*)(src + (size_t)U * 16),
                                       (lds_void_t*)(dst + (size_t)(i * 256 + wbase) * 16), 16, 0, POLICY);
  }
}

// Direct global-to-LDS staging of one RB-byte piece of each of ROWS rows (row
// stride in bytes given at init; with RB a multiple of 128 every wave-wide
// load covers whole cache lines).  LDS rows have a pitch of RB + 16 * PADU
// bytes; units in the padding slots re-read their row's first unit, rows at
// or past nvalid re-read the last valid row, and lanes past the end of the
// block are masked off.  Complete for the workgroup after stage_wait() and a
// barrier.
template <int ROWS, int RB = 128, int PADU = 1>
struct RowStage {
  static constexpr int PITCH = RB + 16 * PADU, NU = RB / 16, PU = NU + PADU, UNITS = ROWS * PU;
  static constexpr int PER = (UNITS + 255) / 256;
  uint32_t off[PER];
  __device__ __forceinline__ void init(int64_t stride, int nvalid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int U = i * 256 + (int)threadIdx.x;
      int r = U / PU;
      const int u = U % PU;
      if (r > nvalid - 1) r = nvalid - 1;
      off[i] = (uint32_t)(r * stride + (u < NU ? u : 0) * 16);
    }
  }
  __device__ __forceinline__ void issue(const unsigned char* src, unsigned char* dst) const {
    const int wbase = (int)(threadIdx.x & ~63u);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      if (UNITS % 256 == 0 || i + 1 < PER || i * 256 + (int)threadIdx.x < UNITS) {
        uint32_t o = off[i];
        asm volatile("" : "+v"(o));
        __builtin_amdgcn_global_load_lds((gbl_void_t*)(src + o),
                                         (lds_void_t*)(dst + (size_t)(i * 256 + wbase) * 16), 16, 0, 0);
      }
    }
  }
};

// A bf16 32x32x16 operand fragment whose contraction index runs down the rows
// of a row-major 16-bit matrix X in LDS (row pitch in bytes, a multiple of 8):
// lane (n = l%32, h = l/32) receives X[r0 + 8h + t][c0 + n], t < 8 (c0 a
// multiple of 4).  Two transposing LDS reads: in each, lane 4j + q of a
// 16-lane group names the 8 bytes X[r + j][c + 4q .. c + 4q + 3], and lane m
// of the group receives column c + m of the four rows r .. r + 3.
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

typedef __attribute__((address_space(3))) const unsigned char lds_cu8;

// Padding (16-byte units) after RB bytes of row data that makes the row pitch
// a bank-conflict-free layout for lds_frag_rows.  LDS has 64 four-byte banks
// and serves a transposing 8-byte read 32 lanes at a time; those lanes read
// 16 consecutive dwords of each of 4 consecutive rows, which land on disjoint
// banks when the pitch is 16 or 48 dwords modulo 64.
constexpr int tr_pad_units(int rb) {
  const int d = (rb / 4) % 64;
  const int a = ((16 - d) % 64 + 64) % 64, b = ((48 - d) % 64 + 64) % 64;
  return (a < b ? a : b) / 4;
}
static_assert(tr_pad_units(512) == 4 && tr_pad_units(128) == 4 && tr_pad_units(64) == 0 &&
              tr_pad_units(256) == 4 && tr_pad_units(32) == 2, "transposing-read pitches");

__device__ __forceinline__ bf16x8 lds_frag_rows(lds_cu8* X, int pitch, int r0, int c0) {
  const int l = threadIdx.x & 63, g = l >> 4, j = (l >> 2) & 3, q = l & 3;
  lds_cu8* p = X + (r0 + 8 * (g >> 1) + j) * pitch + (c0 + 16 * (g & 1) + 4 * q) * 2;
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + 4 * pitch));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

__device__ __forceinline__ bf16x8 lds_frag_rows(const unsigned char* X, int pitch, int r0, int c0) {
  const int l = threadIdx.x & 63, g = l >> 4, j = (l >> 2) & 3, q = l & 3;
  const unsigned char* p = X + (r0 + 8 * (g >> 1) + j) * pitch + (c0 + 16 * (g & 1) + 4 * q) * 2;
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + 4 * pitch));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Wait for this thread's outstanding global loads, the LDS stages included.
__device__ __forceinline__ void stage_wait() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// s_waitcnt immediate that waits until at most N vector memory operations of
// this thread are outstanding (N < 64; expcnt and lgkmcnt not waited for).
// Operations retire in issue order, so every one issued before the N youngest
// has completed.
constexpr int vmcnt_imm(int N) { return (N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

// Edge attributes of edge (i <- j) from the node attribute rows v_i, v_j
// (dim + 1 values each): concat [p_i, p_j, s_i, s_j] or diff v_i - v_j,
// zero-padded to 8 (Sec. 2.1).
template <typename V>
__device__ __forceinline__ void edge_attr_rows(const V& vi, const V& vj, int dim, int mode, float x[8]) {
#pragma unroll
  for (int c = 0; c < 8; ++c) x[c] = 0.0f;
  if (dim == 2) {
    if (mode == DSMP_ATTR_CONCAT) {
      x[0] = vi[0]; x[1] = vi[1]; x[2] = vj[0]; x[3] = vj[1]; x[4] = vi[2]; x[5] = vj[2];
    } else {
      x[0] = vi[0] - vj[0]; x[1] = vi[1] - vj[1]; x[2] = vi[2] - vj[2];
    }
  } else {
    if (mode == DSMP_ATTR_CONCAT) {
      x[0] = vi[0]; x[1] = vi[1]; x[2] = vi[2]; x[3] = vj[0]; x[4] = vj[1]; x[5] = vj[2];
      x[6] = vi[3]; x[7] = vj[3];
    } else {
      x[0] = vi[0] - vj[0]; x[1] = vi[1] - vj[1]; x[2] = vi[2] - vj[2]; x[3] = vi[3] - vj[3];
    }
  }
}

__device__ __forceinline__ void edge_attr(const float* __restrict__ na, int dim, int mode, int i, int j,
                                          float x[8]) {
  edge_attr_rows(na + (size_t)i * (dim + 1), na + (size_t)j * (dim + 1), dim, mode, x);
}

// Workgroup barrier for LDS traffic only: the workgroup's LDS writes are
// complete and visible after it, while global loads issued before it stay
// in flight (a full __syncthreads() waits for them as well).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Workgroup barrier that waits for this wave's LDS instructions alone
// (lgkmcnt): global loads, stores and global-to-LDS copies in flight stay in
// flight, so a caller that reads copied data waits for those copies itself
// (vmcnt) before it.  Even lds_barrier() waits for every outstanding vector
// memory operation once global-to-LDS copies are in flight (its LDS fence
// covers them), stores included.  The empty asm statements keep the compiler
// from moving memory accesses across the barrier.
__device__ __forceinline__ void lds_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0); vmcnt and expcnt not waited for
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Pre-activation of the first kernel-MLP layer for one output: b1 + W1 x as
// a chain of fused multiply-adds in attribute order (w: the 8 weights of the
// output, zero past de).
__device__ __forceinline__ float layer1_pre(const float* __restrict__ w, float b, const float x[8]) {
  const f32x4 wa = *reinterpret_cast<const f32x4*>(w);
  const f32x4 wb = *reinterpret_cast<const f32x4*>(w + 4);
  float v = b;
  v = __builtin_fmaf(wa[0], x[0], v); v = __builtin_fmaf(wa[1], x[1], v);
  v = __builtin_fmaf(wa[2], x[2], v); v = __builtin_fmaf(wa[3], x[3], v);
  v = __builtin_fmaf(wb[0], x[4], v); v = __builtin_fmaf(wb[1], x[5], v);
  v = __builtin_fmaf(wb[2], x[6], v); v = __builtin_fmaf(wb[3], x[7], v);
  return v;
}

// Attribute slots that can be nonzero for an attribute mode and dimension
// (the layouts of edge_attr_rows).
__host__ __device__ inline int attr_slots(int dim, int mode) {
  return mode == DSMP_ATTR_DIFF ? 4 : (dim == 2 ? 6 : 8);
}

// ReLU as one integer maximum over the bits: a positive float is a positive
// signed integer and keeps its bits; +0, -0 and every negative float give +0.
// Equal to (v > 0 ? v : +0) for every value that is not a NaN.
__device__ __forceinline__ float relu_bits(float v) {
  const int i = __float_as_int(v);
  return __int_as_float(i > 0 ? i : 0);
}

// v where bit `bit` of `word` is set, else +0: the bit, sign-extended to a
// whole word (one bit-field extract, inline assembly so that it is not
// turned back into a compare and select), masks the float's bits.  The
// assembly reads only the mask word; v, which may be a matrix-core result,
// goes through an ordinary AND.
__device__ __forceinline__ float keep_if_bit(float v, uint32_t word, int bit) {
  int m;
  asm("v_bfe_i32 %0, %1, %2, 1" : "=v"(m) : "v"(word), "i"(bit));
  return __int_as_float(__float_as_int(v) & m);
}

// ReLU of v, with its mask bit [v > 0] ORed into position `bit` of `word`.
// The bit is a clamp of the ReLU output's bits to [0, 1], one vector
// instruction that leaves no lane mask in scalar registers to keep live.  It
// is inline assembly and reads the ReLU output, never v itself: v may be a
// matrix-core result, and the wait states the compiler inserts before the
// first vector read of such a result are not applied to inline assembly.
__device__ __forceinline__ float relu_mask(float v, uint32_t& word, int bit) {
  const float z = relu_bits(v);
  int r;
  asm("v_med3_i32 %0, %1, 0, 1" : "=v"(r) : "v"(__float_as_int(z)));
  word |= (uint32_t)r << bit;
  return z;
}

// p[0] + p[stride] + ... + p[(n-1) stride], added in index order starting
// from +0 (the same bits as the plain loop), with the loads issued eight at a
// time ahead of their additions instead of one load-wait-add per term.
__device__ __forceinline__ float ordered_sum(const float* __restrict__ p, int64_t stride, int n) {
  float s = 0.0f;
  for (int c0 = 0; c0 < n; c0 += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = c0 + u < n ? p[(int64_t)(c0 + u) * stride] : 0.0f;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (c0 + u < n) s += v[u];
  }
  return s;
}

// A DL x DL fp32 matrix (16-byte aligned) into LDS rows of pitch DL + 1 by a
// 256-thread workgroup, every load issued before the first LDS write.
template <int DL>
__device__ __forceinline__ void stage_square(float (*dst)[DL + 1], const float* __restrict__ src) {
  constexpr int N4 = DL * DL / 4 / 256;
  static_assert(N4 >= 1 && DL * DL % 1024 == 0, "whole float4 per thread");
  float4 v[N4];
#pragma unroll
  for (int u = 0; u < N4; ++u) v[u] = reinterpret_cast<const float4*>(src)[threadIdx.x + 256 * u];
#pragma unroll
  for (int u = 0; u < N4; ++u) {
    const int e = 4 * (threadIdx.x + 256 * u), r = e / DL, c = e % DL;
    dst[r][c] = v[u].x;
    dst[r][c + 1] = v[u].y;
    dst[r][c + 2] = v[u].z;
    dst[r][c + 3] = v[u].w;
  }
}

// Byte offsets of the sections of a packed parameter buffer.
struct PackLayout {
  size_t w1l, b1l, w2p, b2, w3f, w3q, w3t, b3t, b3n, w2t, wr, br, wgt, wht, w3u, total;
};

inline PackLayout pack_layout(int d, int h1, int h2, int esz) {
  PackLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    off = (off + 255) & ~size_t(255);
    size_t o = off;
    off += bytes;
    return o;
  };
  L.w1l = take((size_t)h1 * 8 * 4);           // fp32 [2][h1/2][8]
  L.b1l = take((size_t)h1 * 4);               // fp32 [2][h1/2]
  L.w2p = take((size_t)h2 * h1 * esz);        // T [h2][h1 permuted]
  L.b2 = take((size_t)h2 * 4);                // fp32 [h2]
  L.w3f = take((size_t)d * d * h2 * esz);     // T [p][q][h2 permuted]
  L.w3q = take((size_t)d * d * h2 * esz);     // T [q][p][h2 permuted]
  L.w3t = take((size_t)d * h2 * d * esz);     // T [p][k][q]
  L.b3t = take((size_t)d * d * esz);          // T [q][p]
  L.b3n = take((size_t)d * d * esz);          // T [p][q]
  L.w2t = take((size_t)h1 * h2 * esz);        // T [j][h2 permuted]
  L.wr = take((size_t)d * d * 4);             // fp32 [q][p] (rounded to the layer dtype)
  L.br = take((size_t)d * 4);                 // fp32 [d]
  // W3~ for the aggregate form, in the segment-sum K order (K = h2*d + d):
  // (+128: the GEMM reads rows in whole 128-byte pieces)
  L.wgt = take((size_t)d * (h2 + 1) * d * esz + 128);   // T [q][K(k, p)]
  L.wht = take((size_t)d * (h2 + 1) * d * esz + 128);   // T [p][K(k, q)]
  L.w3u = take((size_t)h2 * d * d * esz);         // T [k*d + p][q] (U GEMM of the aggregate dz)
  L.total = (off + 255) & ~size_t(255);
  return L;
}

// Edges per workgroup tile of the edge kernels (4 waves x 2 tiles x 32).
constexpr int EDGE_TILE = 256;

enum { MODE_FWD = 0, MODE_DH = 1, MODE_MLP = 2 };

// Arguments of the edge contraction (forward messages, or the feature
// gradient when run over the edges in source order).
struct EdgeArgs {
  int64_t E, n_dst, n_src;
  const int32_t* row_ptr;
  const int32_t* col;
  const int32_t* dst;
  const int32_t* csc_ptr;
  const int32_t* csc_eid;
  const float* node_attr;
  int dim, attr_mode;
  const unsigned char* gath;     // FWD: h_in [n_src][d]; DH: g [n_dst][d]  (layer dtype)
  const unsigned char* packed;
  PackLayout L;
  unsigned char* zE;             // [E][h2] layer dtype: FWD writes (if set), DH reads
  unsigned char* z1E;            // [E][h1] layer dtype: FWD writes (if set)
  unsigned char* zmask;          // [E][(h1+h2)/8] ReLU mask bits of z1 and z: FWD writes (if set)
  unsigned char* xE;             // [E][16] bf16 edge attributes, high then low parts: FWD writes (if set)
  float* out_direct;             // [segments][d]
  float* out_part;               // [tiles][2][d]
};

dsmp_status launch_edge_contract(dsmp_handle* h, const dsmp_layer_desc& desc, int mode,
                                 const EdgeArgs& a);

// Per-layer buffer the forward fills for the backward: y [n_dst][d] fp32,
// z [E][h2] and z1 [E][h1] in the layer dtype and the permuted order, their
// ReLU mask bits [E][(h1+h2)/8], the per-destination sums S [n_dst][(h2+1)d]
// of the aggregate form, and (bf16 layers) the edge attributes split into
// bf16 high and low parts [E][16] for the dW1 product.
struct SavedLayout {
  size_t y, zE, z1E, zmask, os, xE, total;
};
SavedLayout saved_layout(const dsmp_layer_desc& d, int64_t n_dst, int64_t E);
size_t fwd_ws_bytes(const dsmp_layer_desc& d, int64_t n_dst, int64_t E);
dsmp_status check_layer_desc(dsmp_handle* h, const dsmp_layer_desc* d);
dsmp_status check_graph(dsmp_handle* h, const dsmp_graph* g, bool need_csc);
int layer_attr_width(const dsmp_layer_desc& d);

// Whether the backward of an aggregate-form layer runs the fused edge-gradient
// pass (bf16, h1 = h2 in {64, 128}, d in {32, 64}).  That pass recomputes z1
// and the edge attributes, so the forward then stores neither.
bool fused_edge_grads(const dsmp_layer_desc& d);
// bf16 aggregate layers at d = 128, h1 = h2 = 256: dz with the feature-gradient
// terms in one pass, da1 with the dW1 sums, dW2 with z1 recomputed
bool dz_with_m(const dsmp_layer_desc& d, bool agg);

// Aggregate form of the edge contraction (nnconv_agg.hip).
bool use_aggregate(const dsmp_handle* h, const dsmp_layer_desc& d, int64_t n_dst, int64_t E);
int64_t agg_ktot(const dsmp_layer_desc& d);
int agg_gemm_slices(int64_t n_rows, const dsmp_layer_desc& d);
int agg_dw3_slices(int64_t n_rows);
dsmp_status launch_outer_sum(dsmp_handle* h, const dsmp_layer_desc& d, int64_t n_seg, const int32_t* seg_ptr,
                             const int32_t* pos_eid, const int32_t* row_of, const unsigned char* zE,
                             const unsigned char* u, unsigned char* out);
dsmp_status launch_w3_gemm(dsmp_handle* h, const dsmp_layer_desc& d, int64_t n_rows, const unsigned char* A,
                           const unsigned char* BT, int nsl, float* part);
dsmp_status launch_dw3_agg(dsmp_handle* h, const dsmp_layer_desc& d, int64_t n_rows, const unsigned char* OS,
                           const unsigned char* G, float* part, float* dW3, float* db3, int accumulate);

}  // namespace dsmp
