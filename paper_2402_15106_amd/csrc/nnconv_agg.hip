// Aggregate-first evaluation of the NNConv edge contraction (eq. (1)).
//
// The message of edge e = (i <- j) is bilinear in the kernel-MLP output z_e
// and the source row h_j:
//     m_e[q] = sum_{k,p} W3[p*d+q][k] z_e[k] h_j[p] + sum_p b3[p*d+q] h_j[p].
// The mean over the edges of i is linear, so with z~ = [z; 1]
//     agg_i[q] = (1/deg_i) sum_{k,p} W3~[p*d+q][k] S_i[k][p],
//     S_i[k][p] = sum_{e in in(i)} z~_e[k] h_j(e)[p],
// one GEMM over the per-destination sums S (n_dst x (h2+1)d) in place of one
// product per edge.  The feature gradient has the same form over the edges
// leaving a source j, with T_j[k][q] = sum_{e in out(j)} z~_e[k] g_e[q] and
// dh_j[p] = sum_{k,q} W3~[p*d+q][k] T_j[k][q]; the weight gradient is
// dW3[p*d+q][k] = sum_i g_i[q] S_i[k][p] (g_e = g_i for every edge into i).
// Neither form writes anything of size E x d x d.
//
// K order of a sum row.  The (h2/32) x (d/32) tiles of 32 x 32 are stored in
// MFMA accumulator order: tile t = kt*(d/32) + ct, lane l, register r at
// K = 1024 t + 16 l + r holds k = 32 kt + 8 (r/4) + 4 (l/32) + r%4 (the
// stored, permuted z order) and c = 32 ct + l%32; the d values of the z~ = 1
// row follow at K = h2*d + c.  The packed W3 matrices (WgT, WhT) use the same
// K order, so neither side is ever transposed in memory.
#include "nnconv.hpp"

using namespace dsmp;

namespace {

template <typename T>
__device__ __forceinline__ typename MT<T>::frag ldf(const void* p) {
  return *reinterpret_cast<const typename MT<T>::frag*>(p);
}

// Copy 4 gathered rows (16-byte unit kg of each) into LDS transposed: row
// (element) kg*KPU + w, columns c0..c0+3.  Null row pointers give zeros.
template <typename T, int ROWB>
__device__ __forceinline__ void put4_transposed(const unsigned char* const r[4], int kg, int c0,
                                                unsigned char* __restrict__ dstl) {
  constexpr int ESZ = sizeof(T);
  uint4 v[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    v[i] = r[i] ? *reinterpret_cast<const uint4*>(r[i] + kg * 16) : make_uint4(0, 0, 0, 0);
  const uint32_t* d0 = reinterpret_cast<const uint32_t*>(&v[0]);
  const uint32_t* d1 = reinterpret_cast<const uint32_t*>(&v[1]);
  const uint32_t* d2 = reinterpret_cast<const uint32_t*>(&v[2]);
  const uint32_t* d3 = reinterpret_cast<const uint32_t*>(&v[3]);
  if constexpr (ESZ == 2) {
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      const int sh = (w & 1) * 16, dw = w >> 1;
      const uint32_t lo = ((d0[dw] >> sh) & 0xFFFFu) | (((d1[dw] >> sh) & 0xFFFFu) << 16);
      const uint32_t hi = ((d2[dw] >> sh) & 0xFFFFu) | (((d3[dw] >> sh) & 0xFFFFu) << 16);
      *reinterpret_cast<uint2*>(dstl + (kg * 8 + w) * ROWB + c0 * ESZ) = make_uint2(lo, hi);
    }
  } else {
#pragma unroll
    for (int w = 0; w < 4; ++w)
      *reinterpret_cast<uint4*>(dstl + (kg * 4 + w) * ROWB + c0 * ESZ) = make_uint4(d0[w], d1[w], d2[w], d3[w]);
  }
}

// ------------------------------------------------------------ segment sums

struct OuterArgs {
  int64_t n_seg;               // segments: destinations (S) or sources (T)
  const int32_t* seg_ptr;      // [n_seg + 1] positions of each segment's edges
  const int32_t* pos_eid;      // NULL: edge id = position; else edge id = pos_eid[position]
  const int32_t* row_of;       // gathered row of edge e
  const unsigned char* zE;     // [E][h2] layer dtype, stored order
  const unsigned char* u;      // gathered rows [*][d] layer dtype
  unsigned char* out;          // [n_seg][ktot] layer dtype
};

template <typename T, int DL, int H2>
struct OuterShape {
  static constexpr int KS = MT<T>::KS, EPL = MT<T>::EPL, ESZ = sizeof(T);
  static constexpr int ECH = 64;                          // edges per staged chunk
  static constexpr int NKT = H2 / 32, NCT = DL / 32, NTILE = NKT * NCT, TPW = (NTILE + 3) / 4;
  static constexpr int ROWB = (ECH + 16 / ESZ) * ESZ;     // LDS row pitch (bytes)
  static constexpr int ZU = (ECH / 4) * (H2 * ESZ / 16);  // transposed staging units
  static constexpr int UU = (ECH / 4) * (DL * ESZ / 16);
  static constexpr int LDS = (H2 + DL) * ROWB;
  static constexpr int64_t KTOT = (int64_t)H2 * DL + DL;
};

// One workgroup per segment: stage up to 64 of its edges at a time, z~ and
// the gathered rows both transposed to [element][edge], and accumulate the
// outer-product sum tile by tile on MFMA (edges are the contraction index).
template <typename T, int DL, int H2>
__global__ __launch_bounds__(256) void k_outer_sum(OuterArgs a) {
  using S = OuterShape<T, DL, H2>;
  using M = MT<T>;
  constexpr int KS = S::KS, EPL = S::EPL, ESZ = S::ESZ, ECH = S::ECH;
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* zt = smem;
  unsigned char* ut = smem + H2 * S::ROWB;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  const int64_t n = blockIdx.x;
  const int64_t pa = a.seg_ptr[n], pb = a.seg_ptr[n + 1];

  f32x16 acc[S::TPW];
#pragma unroll
  for (int j = 0; j < S::TPW; ++j) acc[j] = f32x16{};
  float hs = 0.0f;   // z~ = 1 row: sum of the gathered rows (threads tid < DL)

  for (int64_t c0 = pa; c0 < pb; c0 += ECH) {
    const int cnt = (int)(pb - c0 < ECH ? pb - c0 : ECH);
    __syncthreads();   // previous chunk fully consumed
    for (int x = tid; x < S::ZU + S::UU; x += 256) {
      const bool isz = x < S::ZU;
      const int y = isz ? x : x - S::ZU;
      const int eq = y % (ECH / 4), kg = y / (ECH / 4);
      const unsigned char* r[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int sl = 4 * eq + i;
        r[i] = nullptr;
        if (sl < cnt) {
          const int64_t pos = c0 + sl;
          const int64_t e = a.pos_eid ? (int64_t)a.pos_eid[pos] : pos;
          r[i] = isz ? a.zE + (size_t)e * H2 * ESZ : a.u + (size_t)a.row_of[e] * DL * ESZ;
        }
      }
      if (isz) put4_transposed<T, S::ROWB>(r, kg, 4 * eq, zt);
      else put4_transposed<T, S::ROWB>(r, kg, 4 * eq, ut);
    }
    __syncthreads();
    const int nks = (cnt + KS - 1) / KS;
    for (int ks = 0; ks < nks; ++ks) {
      const int col = (ks * KS + hh * EPL) * ESZ;
#pragma unroll
      for (int j = 0; j < S::TPW; ++j) {
        const int ti = wv + 4 * j;
        if (ti < S::NTILE) {
          const int kt = ti / S::NCT, ct = ti % S::NCT;
          const auto A = ldf<T>(zt + (kt * 32 + l32) * S::ROWB + col);
          const auto B = ldf<T>(ut + (ct * 32 + l32) * S::ROWB + col);
          acc[j] = M::mma(A, B, acc[j]);
        }
      }
    }
    if (tid < DL) {
      const T* row = reinterpret_cast<const T*>(ut + tid * S::ROWB);
      for (int s = 0; s < cnt; ++s) hs += (float)row[s];
    }
  }

  unsigned char* o = a.out + (size_t)n * S::KTOT * ESZ;
#pragma unroll
  for (int j = 0; j < S::TPW; ++j) {
    const int ti = wv + 4 * j;
    if (ti < S::NTILE) {
      unsigned char* dst = o + ((size_t)ti * 1024 + lane * 16) * ESZ;
      if constexpr (ESZ == 2) {
        float v[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = acc[j][r];
        *reinterpret_cast<bf16x8*>(dst) = pack_frag<__bf16>(v);
        *reinterpret_cast<bf16x8*>(dst + 16) = pack_frag<__bf16>(v + 8);
      } else {
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4)
          *reinterpret_cast<f32x4*>(dst + r4 * 16) =
              f32x4{acc[j][4 * r4], acc[j][4 * r4 + 1], acc[j][4 * r4 + 2], acc[j][4 * r4 + 3]};
      }
    }
  }
  if (tid < DL) reinterpret_cast<T*>(o)[(size_t)H2 * DL + tid] = (T)hs;
}

// bf16: the chunk's rows of z~ and of the gathered rows are copied to LDS as
// they are (each wave-wide load covers four whole z rows or eight gathered
// rows), and the fragments, whose contraction index is the edge, come from
// transposing LDS reads.  Slots past the segment's last edge re-read its last
// edge and are zeroed in the A fragment.
template <int DL, int H2>
struct OuterTrShape {
  static constexpr int ECH = 64;
  static constexpr int ZPAD = tr_pad_units(H2 * 2), UPAD = tr_pad_units(DL * 2);
  static constexpr int ZP = H2 * 2 + 16 * ZPAD, UP = DL * 2 + 16 * UPAD;   // LDS row pitches
  static constexpr int ZNU = H2 * 2 / 16, UNU = DL * 2 / 16;   // 16-byte units per row
  static constexpr int ZU = ECH * (ZNU + ZPAD), UU = ECH * (UNU + UPAD);
  static constexpr int NKT = H2 / 32, NCT = DL / 32, NTILE = NKT * NCT, TPW = (NTILE + 3) / 4;
  static constexpr int LDS = ECH * (ZP + UP);
  static constexpr int64_t KTOT = (int64_t)H2 * DL + DL;
};

template <int DL, int H2, bool AHEAD, int NW = 4>
__global__ __launch_bounds__(64 * NW) void k_outer_sum_tr(OuterArgs a) {
  using S = OuterTrShape<DL, H2>;
  using M = MT<__bf16>;
  constexpr int ECH = S::ECH, NT = 64 * NW, TPW = (S::NTILE + NW - 1) / NW;   // threads, tiles per wave
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int rz[ECH], ru[ECH];   // source rows of the chunk's z and gathered rows
  unsigned char* zl = smem;
  unsigned char* ul = smem + ECH * S::ZP;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5;
  const int64_t G = gridDim.x;
  // AHEAD: workgroup b takes segments b, b + G, ..., and the next segment's
  // bounds, edge ids and gathered-row ids are read while this segment's rows
  // are copied and multiplied, so that a segment waits for the copy of its
  // rows alone, not for the chain of index reads ahead of it.  Otherwise
  // workgroup b takes segment b alone (G = n_seg).
  // Slot tid < ECH of a chunk takes the chunk's edge min(tid, cnt - 1).
  auto slot_pos = [&](int64_t c0, int64_t end) {
    const int cnt = (int)(end - c0 < ECH ? end - c0 : ECH);
    return c0 + (tid < cnt ? tid : cnt - 1);
  };
  int64_t n = blockIdx.x, pa = 0, pb = 0;
  int pz = 0, pu = 0;   // first chunk of segment n: edge id and gathered row of slot tid
  if (n < a.n_seg) {
    pa = a.seg_ptr[n];
    pb = a.seg_ptr[n + 1];
    if (AHEAD && tid < ECH && pb > pa) {
      const int64_t pos = slot_pos(pa, pb);
      pz = a.pos_eid ? a.pos_eid[pos] : (int)pos;
      pu = a.row_of[pz];
    }
  }
  for (; n < a.n_seg; n += G) {
    // the next segment's bounds (an empty range past the last segment)
    const int64_t nn = AHEAD ? n + G : a.n_seg;
    const int64_t qa = AHEAD ? a.seg_ptr[nn < a.n_seg ? nn : a.n_seg] : 0;
    const int64_t qb = AHEAD ? a.seg_ptr[nn < a.n_seg ? nn + 1 : a.n_seg] : 0;
    f32x16 acc[TPW];
#pragma unroll
    for (int j = 0; j < TPW; ++j) acc[j] = f32x16{};
    float hs = 0.0f;   // z~ = 1 row: sum of the gathered rows (threads tid < DL)
    const bool ahead = AHEAD && tid < ECH && qb > qa;   // this thread reads ahead a slot of the next segment
    for (int64_t c0 = pa; c0 < pb; c0 += ECH) {
      const int cnt = (int)(pb - c0 < ECH ? pb - c0 : ECH);
      const bool first = c0 == pa;
      __syncthreads();   // previous chunk fully consumed
      if (tid < ECH) {
        int z = pz, u = pu;
        if (!AHEAD || !first) {
          const int64_t pos = slot_pos(c0, pb);
          z = a.pos_eid ? a.pos_eid[pos] : (int)pos;
          u = a.row_of[z];
        }
        rz[tid] = z;
        ru[tid] = u;
      }
      if (first && ahead) {   // the next segment's edge ids, in flight with this chunk's copy
        const int64_t pos = slot_pos(qa, qb);
        pz = a.pos_eid ? a.pos_eid[pos] : (int)pos;
      }
      __syncthreads();
      const int wbase = tid & ~63;
      for (int U0 = 0; U0 < S::ZU; U0 += NT) {
        const int U = U0 + tid, r = U / (S::ZNU + S::ZPAD), u = U % (S::ZNU + S::ZPAD);
        if (U < S::ZU)
          __builtin_amdgcn_global_load_lds(
              (gbl_void_t*)(a.zE + (size_t)rz[r < ECH ? r : ECH - 1] * H2 * 2 + (u < S::ZNU ? u : 0) * 16),
              (lds_void_t*)(zl + (size_t)(U0 + wbase) * 16), 16, 0, 0);
      }
      for (int U0 = 0; U0 < S::UU; U0 += NT) {
        const int U = U0 + tid, r = U / (S::UNU + S::UPAD), u = U % (S::UNU + S::UPAD);
        if (U < S::UU)
          __builtin_amdgcn_global_load_lds(
              (gbl_void_t*)(a.u + (size_t)ru[r < ECH ? r : ECH - 1] * DL * 2 + (u < S::UNU ? u : 0) * 16),
              (lds_void_t*)(ul + (size_t)(U0 + wbase) * 16), 16, 0, 0);
      }
      stage_wait();
      __syncthreads();
      if (first && ahead) pu = a.row_of[pz];   // in flight with this chunk's products
      const int nks = (cnt + 15) / 16;
      for (int ks = 0; ks < nks; ++ks) {
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
          const int ti = wv + NW * j;
          if (ti < S::NTILE) {
            const int kt = ti / S::NCT, ct = ti % S::NCT;
            bf16x8 A = lds_frag_rows(zl, S::ZP, ks * 16, kt * 32);
            if (ks * 16 + 16 > cnt) {   // slots past the last edge
#pragma unroll
              for (int t = 0; t < 8; ++t)
                if (ks * 16 + 8 * hh + t >= cnt) A[t] = (__bf16)0.0f;
            }
            acc[j] = M::mma(A, lds_frag_rows(ul, S::UP, ks * 16, ct * 32), acc[j]);
          }
        }
      }
      if (tid < DL)
        for (int e = 0; e < cnt; ++e) hs += (float)*reinterpret_cast<const __bf16*>(ul + e * S::UP + tid * 2);
    }
    if (pb <= pa && ahead) {   // a segment with no edges: nothing to overlap with
      const int64_t pos = slot_pos(qa, qb);
      pz = a.pos_eid ? a.pos_eid[pos] : (int)pos;
      pu = a.row_of[pz];
    }

    unsigned char* o = a.out + (size_t)n * S::KTOT * 2;
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
      const int ti = wv + NW * j;
      if (ti < S::NTILE) {
        unsigned char* dst = o + ((size_t)ti * 1024 + lane * 16) * 2;
        float v[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = acc[j][r];
        *reinterpret_cast<bf16x8*>(dst) = pack_frag<__bf16>(v);
        *reinterpret_cast<bf16x8*>(dst + 16) = pack_frag<__bf16>(v + 8);
      }
    }
    if (tid < DL) reinterpret_cast<__bf16*>(o)[(size_t)H2 * DL + tid] = (__bf16)hs;
    if (!AHEAD) break;
    pa = qa;
    pb = qb;
  }
}

// ------------------------------------------------------------ GEMM with W3~

struct GemmArgs {
  int64_t n_rows, ktot;
  const unsigned char* A;    // [n_rows][ktot] layer dtype (segment sums)
  const unsigned char* BT;   // [DL][ktot] layer dtype (packed W3~ in the sum order)
  int nsl;                   // K slices
  int64_t csl;               // K chunks per slice
  float* part;               // [nsl][n_rows][DL] partial products
};

template <typename T, int DL>
struct GemmShape {
  static constexpr int ESZ = sizeof(T), KS = MT<T>::KS;
  static constexpr int CB = 128, SPC = CB / (KS * ESZ);   // bytes of a row per chunk, K steps per chunk
  static constexpr int AB = 128 * RowStage<128>::PITCH, BB = DL * RowStage<DL>::PITCH;
  static constexpr int BUF = AB + BB, LDS = 2 * BUF;
};

// part[s][n][c] = sum over slice s of K:  A[n][K] * BT[c][K].  A workgroup
// owns 128 rows (32 per wave) and all d columns of one K slice.  K advances
// in chunks of 128 bytes per row: the chunk of the 128 A rows and the d BT
// rows is copied to LDS by whole cache lines while the previous chunk is
// multiplied (two buffers).
template <typename T, int DL>
__global__ __launch_bounds__(256) void k_w3_gemm(GemmArgs a) {
  using M = MT<T>;
  using G = GemmShape<T, DL>;
  constexpr int KS = M::KS, EPL = M::EPL, ESZ = sizeof(T), NCT = DL / 32, SPC = G::SPC;
  constexpr int PITCH = RowStage<128>::PITCH;
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  const int64_t r0 = (int64_t)blockIdx.x * 128;
  const int s = blockIdx.y;
  const int64_t nstep = a.ktot / KS, nchunk = (nstep + SPC - 1) / SPC;
  const int64_t c0 = s * a.csl, c1 = c0 + a.csl < nchunk ? c0 + a.csl : nchunk;
  f32x16 acc[NCT];
#pragma unroll
  for (int ct = 0; ct < NCT; ++ct) acc[ct] = f32x16{};
  if (c0 < c1) {   // uniform over the workgroup; an empty slice writes zeros
  const int nvalid = (int)(a.n_rows - r0 < 128 ? a.n_rows - r0 : 128);
  RowStage<128> sa;
  RowStage<DL> sb;
  sa.init(a.ktot * ESZ, nvalid);
  sb.init(a.ktot * ESZ, DL);
  const unsigned char* ga = a.A + (size_t)r0 * a.ktot * ESZ;
  sa.issue(ga + c0 * G::CB, smem);
  sb.issue(a.BT + c0 * G::CB, smem + G::AB);
  stage_wait();
  __syncthreads();
  for (int64_t c = c0; c < c1; ++c) {
    unsigned char* cur = smem + ((c - c0) & 1) * G::BUF;
    if (c + 1 < c1) {
      unsigned char* nxt = smem + ((c + 1 - c0) & 1) * G::BUF;
      sa.issue(ga + (c + 1) * G::CB, nxt);
      sb.issue(a.BT + (c + 1) * G::CB, nxt + G::AB);
    }
    const int nst = (int)(nstep - c * SPC < SPC ? nstep - c * SPC : SPC);
    const unsigned char* la = cur + (wv * 32 + l32) * PITCH + hh * EPL * ESZ;
    const unsigned char* lb = cur + G::AB + l32 * PITCH + hh * EPL * ESZ;
#pragma unroll
    for (int st = 0; st < SPC; ++st) {
      if (st < nst) {
        const auto A = ldf<T>(la + st * KS * ESZ);
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
          acc[ct] = M::mma(A, ldf<T>(lb + ct * 32 * PITCH + st * KS * ESZ), acc[ct]);
      }
    }
    stage_wait();
    __syncthreads();
  }
  }
  float* out = a.part + (size_t)s * a.n_rows * DL;
#pragma unroll
  for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t rr = r0 + wv * 32 + 8 * (r / 4) + 4 * hh + (r % 4);
      if (rr < a.n_rows) out[rr * DL + ct * 32 + l32] = acc[ct][r];
    }
}

// ------------------------------------------------------------ dW3 from S

struct DW3AggArgs {
  int64_t n_rows, ktot, kcols;
  const unsigned char* OS;   // [n_rows][ktot] layer dtype
  const unsigned char* G;    // [n_rows][DL] layer dtype (g_i)
  int nsl;
  int64_t rows_per_sl;       // multiple of 64
  float* part;               // [nsl][DL][kcols]
};

template <typename T, int DL>
struct DW3AggShape {
  static constexpr int KS = MT<T>::KS, EPL = MT<T>::EPL, ESZ = sizeof(T);
  static constexpr int NCH = 64, KR = 256;              // rows per chunk, K columns per workgroup
  static constexpr int NQT = DL / 32, NKT = KR / 32, NTILE = NQT * NKT, TPW = NTILE / 4;
  static constexpr int ROWB = (NCH + 16 / ESZ) * ESZ;
  static constexpr int OU = (NCH / 4) * (KR * ESZ / 16), GU = (NCH / 4) * (DL * ESZ / 16);
  static constexpr int LDS = (KR + DL) * ROWB;
  static_assert(NTILE % 4 == 0, "tiles split over four waves");
};

// part[s][q][K] = sum over the rows of slice s of g[i][q] * S[i][K]: rows of
// S and g staged transposed to [column][row], rows are the contraction index.
template <typename T, int DL>
__global__ __launch_bounds__(256) void k_dw3_agg(DW3AggArgs a) {
  using S = DW3AggShape<T, DL>;
  using M = MT<T>;
  constexpr int KS = S::KS, EPL = S::EPL, ESZ = S::ESZ, NCH = S::NCH;
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* ot = smem;
  unsigned char* gt = smem + S::KR * S::ROWB;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  const int64_t kc0 = (int64_t)blockIdx.x * S::KR;
  const int s = blockIdx.y;
  const int64_t rb = s * a.rows_per_sl;
  const int64_t re = rb + a.rows_per_sl < a.n_rows ? rb + a.rows_per_sl : a.n_rows;
  f32x16 acc[S::TPW];
#pragma unroll
  for (int j = 0; j < S::TPW; ++j) acc[j] = f32x16{};
  for (int64_t c0 = rb; c0 < re; c0 += NCH) {
    const int cnt = (int)(re - c0 < NCH ? re - c0 : NCH);
    __syncthreads();
    for (int x = tid; x < S::OU + S::GU; x += 256) {
      const bool iso = x < S::OU;
      const int y = iso ? x : x - S::OU;
      const int eq = y % (NCH / 4), kg = y / (NCH / 4);
      const unsigned char* r[4];
      // columns past the end of a row (last K block) read as zeros
      const bool inrow = !iso || kc0 + (int64_t)kg * (16 / ESZ) < a.kcols;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int sl = 4 * eq + i;
        r[i] = sl < cnt && inrow
                   ? (iso ? a.OS + ((size_t)(c0 + sl) * a.ktot + kc0) * ESZ : a.G + (size_t)(c0 + sl) * DL * ESZ)
                   : nullptr;
      }
      if (iso) put4_transposed<T, S::ROWB>(r, kg, 4 * eq, ot);
      else put4_transposed<T, S::ROWB>(r, kg, 4 * eq, gt);
    }
    __syncthreads();
    const int nks = (cnt + KS - 1) / KS;
    for (int ks = 0; ks < nks; ++ks) {
      const int col = (ks * KS + hh * EPL) * ESZ;
#pragma unroll
      for (int j = 0; j < S::TPW; ++j) {
        const int ti = wv * S::TPW + j, qt = ti / S::NKT, kt = ti % S::NKT;
        acc[j] = M::mma(ldf<T>(gt + (qt * 32 + l32) * S::ROWB + col), ldf<T>(ot + (kt * 32 + l32) * S::ROWB + col),
                        acc[j]);
      }
    }
  }
  float* out = a.part + (size_t)s * DL * a.kcols;
#pragma unroll
  for (int j = 0; j < S::TPW; ++j) {
    const int ti = wv * S::TPW + j, qt = ti / S::NKT, kt = ti % S::NKT;
    const int64_t kc = kc0 + kt * 32 + l32;
    if (kc < a.kcols)
#pragma unroll
      for (int r = 0; r < 16; ++r) out[(size_t)(qt * 32 + 8 * (r / 4) + 4 * hh + (r % 4)) * a.kcols + kc] = acc[j][r];
  }
}

// bf16 layers: the same sums with chunks of 32 rows of S (a piece of KR K
// columns: 256, or 128 at d = 128, which halves the accumulators per wave and
// measured 1.5x faster there) and of g copied to LDS by whole cache lines,
// two buffers, and the fragments read by transposing LDS reads (rows are the
// contraction index).  Wave w owns TPW consecutive K tiles of one q tile, so
// one g fragment feeds TPW products.  Rows past the slice re-read its last
// row and are zeroed in the g fragment; columns past the end of a row (last
// K block) are read from the next row (or the buffer's tail padding) and
// never stored.
template <int DL>
struct DW3TrShape {
  static constexpr int ECH = 32, KR = DL == 128 ? 128 : 256;
  using SS = RowStage<ECH, KR * 2, tr_pad_units(KR * 2)>;
  using GS = RowStage<ECH, DL * 2, tr_pad_units(DL * 2)>;
  static constexpr int SB = ECH * SS::PITCH, BUF = SB + ECH * GS::PITCH, LDS = 2 * BUF;
  static constexpr int NQT = DL / 32, NKT = KR / 32, TPW = NQT * NKT / 4;
  static_assert(TPW % 4 == 0 || TPW == 2, "K tiles per wave");
};

template <int DL>
__global__ __launch_bounds__(256) void k_dw3_agg_tr(DW3AggArgs a) {
  using S = DW3TrShape<DL>;
  using M = MT<__bf16>;
  constexpr int ECH = S::ECH, TPW = S::TPW;
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  const int64_t kc0 = (int64_t)blockIdx.x * S::KR;
  const int s = blockIdx.y;
  const int64_t rb = s * a.rows_per_sl;
  const int64_t re = rb + a.rows_per_sl < a.n_rows ? rb + a.rows_per_sl : a.n_rows;
  // the wave's tiles: ti = wv*TPW + j  ->  qt = ti / NKT, kt = ti % NKT (one qt per wave)
  const int qt = (wv * TPW) / S::NKT, kt0 = (wv * TPW) % S::NKT;
  f32x16 acc[TPW];
#pragma unroll
  for (int j = 0; j < TPW; ++j) acc[j] = f32x16{};
  if (rb < re) {   // uniform over the workgroup
    const int nch = (int)((re - rb + ECH - 1) / ECH);
    typename S::SS ss;
    typename S::GS sg;
    auto issue = [&](int c, unsigned char* buf) {
      const int64_t r0 = rb + (int64_t)c * ECH;
      const int nv = (int)(re - r0 < ECH ? re - r0 : ECH);
      ss.init(a.ktot * 2, nv);
      sg.init(DL * 2, nv);
      ss.issue(a.OS + ((size_t)r0 * a.ktot + kc0) * 2, buf);
      sg.issue(a.G + (size_t)r0 * DL * 2, buf + S::SB);
    };
    issue(0, smem);
    stage_wait();
    __syncthreads();
    for (int c = 0; c < nch; ++c) {
      const unsigned char* cur = smem + (c & 1) * S::BUF;
      if (c + 1 < nch) issue(c + 1, smem + ((c + 1) & 1) * S::BUF);
      const int64_t r0 = rb + (int64_t)c * ECH;
      const int cnt = (int)(re - r0 < ECH ? re - r0 : ECH);
      for (int ks = 0; ks * 16 < cnt; ++ks) {
        bf16x8 A = lds_frag_rows(cur + S::SB, S::GS::PITCH, ks * 16, qt * 32);
        if (ks * 16 + 16 > cnt) {
#pragma unroll
          for (int t = 0; t < 8; ++t)
            if (ks * 16 + 8 * hh + t >= cnt) A[t] = (__bf16)0.0f;
        }
#pragma unroll
        for (int j = 0; j < TPW; ++j)
          acc[j] = M::mma(A, lds_frag_rows(cur, S::SS::PITCH, ks * 16, (kt0 + j) * 32), acc[j]);
      }
      stage_wait();
      __syncthreads();
    }
  }
  float* out = a.part + (size_t)s * DL * a.kcols;
#pragma unroll
  for (int j = 0; j < TPW; ++j) {
    const int64_t kc = kc0 + (kt0 + j) * 32 + l32;
    if (kc < a.kcols)
#pragma unroll
      for (int r = 0; r < 16; ++r) out[(size_t)(qt * 32 + 8 * (r / 4) + 4 * hh + (r % 4)) * a.kcols + kc] = acc[j][r];
  }
}

// dW3[p*d+q][k] (+)= sum_s part[s][q][K(k, p)], K in the sum order above;
// the bias rows K = h2*d + p give db3[p*d+q].
template <typename T>
__global__ __launch_bounds__(256) void k_dw3_agg_final(int d, int h2, int nsl, const float* __restrict__ part,
                                                       float* __restrict__ dW3, float* __restrict__ db3,
                                                       int accumulate) {
  const int64_t kcols = (int64_t)h2 * d + d, total = (int64_t)d * kcols;
  const int nct = d / 32;
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < total; x += (int64_t)gridDim.x * blockDim.x) {
    // x enumerates (q, K) with K fastest, so the reads of part are contiguous
    const int q = (int)(x / kcols);
    const int64_t K = x % kcols;
    const float v = ordered_sum(part + (int64_t)q * kcols + K, (int64_t)d * kcols, nsl);
    float* o;
    if (K < (int64_t)h2 * d) {
      const int ti = K / 1024, rem = K % 1024, l = rem / 16, r = rem % 16;
      const int kt = ti / nct, ct = ti % nct;
      const int kpos = kt * 32 + 8 * (r / 4) + 4 * (l / 32) + (r % 4), p = ct * 32 + (l % 32);
      o = dW3 + ((int64_t)p * d + q) * h2 + kperm<T>(kpos);
    } else {
      o = db3 + (K - (int64_t)h2 * d) * d + q;
    }
    *o = accumulate ? *o + v : v;
  }
}

// Persistent form of the outer-product sums for few workgroups per CU, with
// the first chunk of the next segment copied while this segment's sums are
// stored.  Loads and stores retire through one in-order counter, so a copy
// issued after a segment's stores would wait for them; here the copy goes out
// first, and the wait at the top of a segment leaves the previous segment's
// stores in flight.  The index chain runs ahead: edge ids two segments ahead,
// gathered-row ids one segment ahead, bounds by scalar loads.  Chunks after a
// segment's first (segments of more than ECH edges) are copied and multiplied
// in turn.  Barriers wait for LDS instructions only (lds_sync: a full
// barrier would wait for the stores).  The products, their order and the stored layout are those of
// k_outer_sum_tr.
template <int DL, int H2, int NW>
__global__ __launch_bounds__(64 * NW) void k_outer_sum_pf(OuterArgs a) {
  using S = OuterTrShape<DL, H2>;
  using M = MT<__bf16>;
  constexpr int ECH = S::ECH, NT = 64 * NW, TPW = (S::NTILE + NW - 1) / NW;
  static_assert(S::NTILE % NW == 0, "every wave holds TPW tiles");
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int rz[ECH], ru[ECH];   // source rows of the chunk's z and gathered rows
  unsigned char* zl = smem;
  unsigned char* ul = smem + ECH * S::ZP;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5;
  const int64_t G = gridDim.x;
  typedef __attribute__((address_space(4))) const int32_t cint32_t;
  cint32_t* sp = (cint32_t*)(a.seg_ptr);
  auto bounds = [&](int64_t n, int64_t& p0, int64_t& p1) {   // empty past the last segment
    const int64_t nc = n < a.n_seg ? n : a.n_seg;
    p0 = sp[nc];
    p1 = n < a.n_seg ? (int64_t)sp[nc + 1] : p0;
  };
  // slot tid < ECH of a chunk takes the chunk's edge min(tid, cnt - 1)
  auto slot_pos = [&](int64_t c0, int64_t end) {
    const int cnt = (int)(end - c0 < ECH ? end - c0 : ECH);
    return c0 + (tid < cnt ? tid : cnt - 1);
  };
  auto edge_of = [&](int64_t pos) -> int { return a.pos_eid ? a.pos_eid[pos] : (int)pos; };
  auto copy_chunk = [&]() {
    const int wbase = tid & ~63;
    for (int U0 = 0; U0 < S::ZU; U0 += NT) {
      const int U = U0 + tid, r = U / (S::ZNU + S::ZPAD), u = U % (S::ZNU + S::ZPAD);
      if (U < S::ZU)
        __builtin_amdgcn_global_load_lds(
            (gbl_void_t*)(a.zE + (size_t)rz[r < ECH ? r : ECH - 1] * H2 * 2 + (u < S::ZNU ? u : 0) * 16),
            (lds_void_t*)(zl + (size_t)(U0 + wbase) * 16), 16, 0, 0);
    }
    for (int U0 = 0; U0 < S::UU; U0 += NT) {
      const int U = U0 + tid, r = U / (S::UNU + S::UPAD), u = U % (S::UNU + S::UPAD);
      if (U < S::UU)
        __builtin_amdgcn_global_load_lds(
            (gbl_void_t*)(a.u + (size_t)ru[r < ECH ? r : ECH - 1] * DL * 2 + (u < S::UNU ? u : 0) * 16),
            (lds_void_t*)(ul + (size_t)(U0 + wbase) * 16), 16, 0, 0);
    }
  };
  f32x16 acc[TPW];
  float hs = 0.0f;   // z~ = 1 row: sum of the gathered rows (threads tid < DL)
  auto multiply = [&](int cnt) {
    const int nks = (cnt + 15) / 16;
    for (int ks = 0; ks < nks; ++ks) {
#pragma unroll
      for (int j = 0; j < TPW; ++j) {
        const int ti = wv + NW * j;
        const int kt = ti / S::NCT, ct = ti % S::NCT;
        bf16x8 A = lds_frag_rows(zl, S::ZP, ks * 16, kt * 32);
        if (ks * 16 + 16 > cnt) {   // slots past the last edge
#pragma unroll
          for (int t = 0; t < 8; ++t)
            if (ks * 16 + 8 * hh + t >= cnt) A[t] = (__bf16)0.0f;
        }
        acc[j] = M::mma(A, lds_frag_rows(ul, S::UP, ks * 16, ct * 32), acc[j]);
      }
    }
    if (tid < DL)
      for (int e = 0; e < cnt; ++e) hs += (float)*reinterpret_cast<const __bf16*>(ul + e * S::UP + tid * 2);
  };

  int64_t n = blockIdx.x;
  if (n >= a.n_seg) return;
  int64_t pa, pb, pa1, pb1, pa2, pb2;
  bounds(n, pa, pb);
  bounds(n + G, pa1, pb1);
  bounds(n + 2 * G, pa2, pb2);
  // the first chunk of segment n, and the ids of segment n + G (and the edge
  // ids of n + 2G) ahead
  int pz1 = 0, pu1 = 0, pz2 = 0;
  if (tid < ECH && pb > pa) {
    const int z = edge_of(slot_pos(pa, pb));
    rz[tid] = z;
    ru[tid] = a.row_of[z];
  }
  if (tid < ECH && pb1 > pa1) pz1 = edge_of(slot_pos(pa1, pb1));
  lds_sync();
  if (pb > pa) copy_chunk();
  if (tid < ECH && pb1 > pa1) pu1 = a.row_of[pz1];
  bool first_iter = true;
  for (; n < a.n_seg; n += G) {
    // the copy of this segment's first chunk; after it only the previous
    // segment's stores (2 TPW per thread) went out
    if (first_iter) stage_wait();
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * TPW));
    first_iter = false;
    lds_sync();
    if (tid < ECH && pb2 > pa2) pz2 = edge_of(slot_pos(pa2, pb2));   // two segments ahead
#pragma unroll
    for (int j = 0; j < TPW; ++j) acc[j] = f32x16{};
    hs = 0.0f;
    if (pb > pa) multiply((int)(pb - pa < ECH ? pb - pa : ECH));
    for (int64_t c0 = pa + ECH; c0 < pb; c0 += ECH) {   // segments of more than ECH edges
      lds_sync();
      if (tid < ECH) {
        const int z = edge_of(slot_pos(c0, pb));
        rz[tid] = z;
        ru[tid] = a.row_of[z];
      }
      lds_sync();
      copy_chunk();
      stage_wait();
      lds_sync();
      multiply((int)(pb - c0 < ECH ? pb - c0 : ECH));
    }
    unsigned char* o = a.out + (size_t)n * S::KTOT * 2;
    // the z~ = 1 row before the next copy, so that exactly 2 TPW stores follow it
    if (tid < DL) reinterpret_cast<__bf16*>(o)[(size_t)H2 * DL + tid] = (__bf16)hs;
    lds_sync();   // every wave is done with the chunk buffers and ids
    if (tid < ECH && pb1 > pa1) {
      rz[tid] = pz1;
      ru[tid] = pu1;
    }
    lds_sync();
    if (pb1 > pa1) copy_chunk();   // segment n + G's first chunk, ahead of this segment's stores
    if (tid < ECH && pb2 > pa2) pu1 = a.row_of[pz2];
    pz1 = pz2;
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
      const int ti = wv + NW * j;
      unsigned char* dst = o + ((size_t)ti * 1024 + lane * 16) * 2;
      float v[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) v[r] = acc[j][r];
      *reinterpret_cast<bf16x8*>(dst) = pack_frag<__bf16>(v);
      *reinterpret_cast<bf16x8*>(dst + 16) = pack_frag<__bf16>(v + 8);
    }
    pa = pa1; pb = pb1;
    pa1 = pa2; pb1 = pb2;
    bounds(n + 3 * G, pa2, pb2);
  }
}

template <typename K>
dsmp_status set_lds_bytes(dsmp_handle* h, K kernel, int bytes) {
  DSMP_HIP(h, hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, bytes));
  return DSMP_OK;
}

template <typename T, int DL, int H2>
dsmp_status outer_shape(dsmp_handle* h, const OuterArgs& a) {
  if constexpr (sizeof(T) == 2) {
    using S = OuterTrShape<DL, H2>;
    // persistent workgroups that read the next segment's indices ahead where
    // fewer than four fit on a CU; with four or more, one segment per
    // workgroup, which lets the dispatcher balance segments of uneven length
    auto ahead = k_outer_sum_tr<DL, H2, true>;
    auto single = k_outer_sum_tr<DL, H2, false>;
    dsmp_status st = set_lds_bytes(h, ahead, S::LDS);
    if (st == DSMP_OK) st = set_lds_bytes(h, single, S::LDS);
    if (st != DSMP_OK) return st;
    int per_cu = 0;
    DSMP_HIP(h, hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, ahead, 256, S::LDS));
    if (per_cu >= 4) {
      hipLaunchKernelGGL(single, dim3((unsigned)a.n_seg), dim3(256), S::LDS, h->stream, a);
    } else {
      // few workgroups fit: eight waves per workgroup, half the tiles per wave,
      // the next segment's first chunk copied ahead of this segment's stores
      auto ahead8 = [] {
        if constexpr (S::NTILE % 8 == 0) return k_outer_sum_pf<DL, H2, 8>;
        else return k_outer_sum_tr<DL, H2, true, 8>;
      }();
      if ((st = set_lds_bytes(h, ahead8, S::LDS)) != DSMP_OK) return st;
      int per_cu8 = 0;
      DSMP_HIP(h, hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu8, ahead8, 512, S::LDS));
      hipLaunchKernelGGL(ahead8,
                         dim3((unsigned)std::min<int64_t>(a.n_seg, (int64_t)h->n_cu * std::max(per_cu8, 1))),
                         dim3(512), S::LDS, h->stream, a);
    }
    DSMP_LAUNCHED(h, "segment outer-product sums");
    return DSMP_OK;
  }
  using S = OuterShape<T, DL, H2>;
  auto kern = k_outer_sum<T, DL, H2>;
  dsmp_status st = set_lds_bytes(h, kern, S::LDS);
  if (st != DSMP_OK) return st;
  hipLaunchKernelGGL(kern, dim3((unsigned)a.n_seg), dim3(256), S::LDS, h->stream, a);
  DSMP_LAUNCHED(h, "segment outer-product sums");
  return DSMP_OK;
}

template <typename T, int DL>
dsmp_status gemm_shape(dsmp_handle* h, const GemmArgs& a) {
  using G = GemmShape<T, DL>;
  auto kern = k_w3_gemm<T, DL>;
  dsmp_status st = set_lds_bytes(h, kern, G::LDS);
  if (st != DSMP_OK) return st;
  hipLaunchKernelGGL(kern, dim3((unsigned)ceil_div(a.n_rows, 128), (unsigned)a.nsl), dim3(256), G::LDS, h->stream, a);
  DSMP_LAUNCHED(h, "W3 GEMM over segment sums");
  return DSMP_OK;
}

template <typename T, int DL>
dsmp_status dw3_shape(dsmp_handle* h, const DW3AggArgs& a) {
  if constexpr (sizeof(T) == 2) {
    using S = DW3TrShape<DL>;
    auto kern = k_dw3_agg_tr<DL>;
    dsmp_status st = set_lds_bytes(h, kern, S::LDS);
    if (st != DSMP_OK) return st;
    hipLaunchKernelGGL(kern, dim3((unsigned)ceil_div(a.kcols, S::KR), (unsigned)a.nsl), dim3(256), S::LDS,
                       h->stream, a);
    DSMP_LAUNCHED(h, "dW3 from segment sums");
    return DSMP_OK;
  }
  using S = DW3AggShape<T, DL>;
  auto kern = k_dw3_agg<T, DL>;
  dsmp_status st = set_lds_bytes(h, kern, S::LDS);
  if (st != DSMP_OK) return st;
  hipLaunchKernelGGL(kern, dim3((unsigned)ceil_div(a.kcols, S::KR), (unsigned)a.nsl), dim3(256), S::LDS, h->stream,
                     a);
  DSMP_LAUNCHED(h, "dW3 from segment sums");
  return DSMP_OK;
}

}  // namespace

namespace dsmp {

int64_t agg_ktot(const dsmp_layer_desc& d) { return (int64_t)d.h2 * d.d + d.d; }

bool use_aggregate(const dsmp_handle* h, const dsmp_layer_desc& d, int64_t n_dst, int64_t E) {
  if (h->edge_algo == DSMP_EDGE_PER_EDGE) return false;
  if (h->edge_algo == DSMP_EDGE_AGGREGATE) return true;
  return n_dst > 0 && E * d.d >= 512 * n_dst;
}

int agg_gemm_slices(int64_t n_rows, const dsmp_layer_desc& d) {
  const int64_t waves = ceil_div(n_rows, 32);
  int nsl = (int)(2048 / (waves > 0 ? waves : 1));
  if (nsl < 1) nsl = 1;
  if (nsl > 16) nsl = 16;
  return nsl;
}

dsmp_status launch_outer_sum(dsmp_handle* h, const dsmp_layer_desc& d, int64_t n_seg, const int32_t* seg_ptr,
                             const int32_t* pos_eid, const int32_t* row_of, const unsigned char* zE,
                             const unsigned char* u, unsigned char* out) {
  if (n_seg == 0) return DSMP_OK;
  OuterArgs a{n_seg, seg_ptr, pos_eid, row_of, zE, u, out};
  if (d.dtype == DSMP_F32) {
    if (d.d == 32) return outer_shape<float, 32, 64>(h, a);
    if (d.d == 64) return outer_shape<float, 64, 128>(h, a);
  } else {
    if (d.d == 32) return outer_shape<__bf16, 32, 64>(h, a);
    if (d.d == 64) return outer_shape<__bf16, 64, 128>(h, a);
    if (d.d == 128) return outer_shape<__bf16, 128, 256>(h, a);
  }
  return fail(h, DSMP_UNSUPPORTED, "unsupported layer shape");
}

dsmp_status launch_w3_gemm(dsmp_handle* h, const dsmp_layer_desc& d, int64_t n_rows, const unsigned char* A,
                           const unsigned char* BT, int nsl, float* part) {
  if (n_rows == 0) return DSMP_OK;
  const int64_t ktot = agg_ktot(d);
  const int esz = d.dtype == DSMP_F32 ? 4 : 2;
  const int64_t nchunk = ceil_div(ktot * esz, 128);
  GemmArgs a{n_rows, ktot, A, BT, nsl, ceil_div(nchunk, nsl), part};
  if (d.dtype == DSMP_F32) {
    if (d.d == 32) return gemm_shape<float, 32>(h, a);
    if (d.d == 64) return gemm_shape<float, 64>(h, a);
  } else {
    if (d.d == 32) return gemm_shape<__bf16, 32>(h, a);
    if (d.d == 64) return gemm_shape<__bf16, 64>(h, a);
    if (d.d == 128) return gemm_shape<__bf16, 128>(h, a);
  }
  return fail(h, DSMP_UNSUPPORTED, "unsupported layer shape");
}

// Row slices of the dW3 product: 16 (at least 64 rows each).  Measured at
// the five workloads, 16 slices were as fast as or faster than 4, 8, 24 and
// 32 (fewer slices cut the partial sums' traffic but leave CUs idle; more add
// partials without speed).
int agg_dw3_slices(int64_t n_rows) {
  int64_t nsl = ceil_div(n_rows, 64);
  if (nsl < 1) nsl = 1;
  if (nsl > 16) nsl = 16;
  return (int)nsl;
}

dsmp_status launch_dw3_agg(dsmp_handle* h, const dsmp_layer_desc& d, int64_t n_rows, const unsigned char* OS,
                           const unsigned char* G, float* part, float* dW3, float* db3, int accumulate) {
  const int nsl = agg_dw3_slices(n_rows);
  const int64_t kcols = agg_ktot(d);
  if (n_rows > 0) {
    DW3AggArgs a{n_rows, agg_ktot(d), kcols, OS, G, nsl, ceil_div(ceil_div(n_rows, nsl), 64) * 64, part};
    dsmp_status st = DSMP_UNSUPPORTED;
    if (d.dtype == DSMP_F32) {
      if (d.d == 32) st = dw3_shape<float, 32>(h, a);
      if (d.d == 64) st = dw3_shape<float, 64>(h, a);
    } else {
      if (d.d == 32) st = dw3_shape<__bf16, 32>(h, a);
      if (d.d == 64) st = dw3_shape<__bf16, 64>(h, a);
      if (d.d == 128) st = dw3_shape<__bf16, 128>(h, a);
    }
    if (st != DSMP_OK) return st;
  }
  const int nuse = n_rows > 0 ? nsl : 0;
  const int64_t total = (int64_t)d.d * kcols;
  unsigned grid = (unsigned)ceil_div(total, 256);
  if (grid > 8192) grid = 8192;
  if (d.dtype == DSMP_F32)
    hipLaunchKernelGGL(k_dw3_agg_final<float>, dim3(grid), dim3(256), 0, h->stream, d.d, d.h2, nuse, part, dW3, db3,
                       accumulate);
  else
    hipLaunchKernelGGL(k_dw3_agg_final<__bf16>, dim3(grid), dim3(256), 0, h->stream, d.d, d.h2, nuse, part, dW3, db3,
                       accumulate);
  DSMP_LAUNCHED(h, "dW3 assembly");
  return DSMP_OK;
}

}  // namespace dsmp
