/*
 * dsmpnn.h -- C ABI of the MI355X (gfx950) hot path of DS-MPNN
 * (Kakka et al., "Sampling-based Distributed Training with Message Passing
 * Neural Network", arXiv 2402.15106).
 *
 * The calls follow the paper's statement of the problem:
 *   sample nodes            (Sec. 2.1; Algorithm 1, node-sampling step)
 *   build the radius graph  (Sec. 2.1; Algorithm 1, edge-index creation and
 *                            edge-sampling steps)
 *   run an edge-conditioned message-passing layer forward and backward
 *                           (eq. (1), eq. (ii); Algorithm 1, graph-convolution
 *                            step with residual, and its backpropagation)
 *
 * Conventions shared by every call
 *   - Pointers marked "device" address GPU memory of the handle's device;
 *     pointers marked "host" address host memory.  The caller owns every
 *     buffer; the library allocates nothing in any call except dsmp_create.
 *   - Work is enqueued on the stream bound with dsmp_set_stream (default:
 *     the null stream) and is asynchronous unless a call says it
 *     synchronises.
 *   - Every call returns a dsmp_status.  On failure nothing has been
 *     enqueued (argument errors are found on the host before any launch),
 *     except where a call states otherwise; dsmp_last_error(h) then holds a
 *     message.  The library never aborts the process.
 *   - Integer index arrays are int32 (sizes beyond 2^31-1 edges or nodes
 *     are rejected with DSMP_UNSUPPORTED).
 *   - Results are deterministic: the same inputs give bitwise-identical
 *     outputs on every run (no floating-point atomics anywhere).
 */
#ifndef DSMPNN_H
#define DSMPNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum dsmp_status {
  DSMP_OK = 0,
  DSMP_INVALID_ARG = 1,          /* a null pointer, a size out of range, ... */
  DSMP_CAPACITY = 2,             /* an output buffer is too small; the needed size is reported */
  DSMP_HIP_ERROR = 3,            /* the HIP runtime reported an error */
  DSMP_UNSUPPORTED = 4,          /* a valid request this build does not implement */
  DSMP_WORKSPACE_TOO_SMALL = 5   /* the workspace passed is smaller than the query said */
} dsmp_status;

typedef struct dsmp_handle dsmp_handle;

/* Version of this ABI (major*10000 + minor*100 + patch). */
int dsmp_version(void);

/* Create a handle bound to HIP device `device` (made current for the calls
 * made through the handle).  *out receives the handle; host memory owned by
 * the library until dsmp_destroy. */
dsmp_status dsmp_create(dsmp_handle** out, int device);
dsmp_status dsmp_destroy(dsmp_handle* h);

/* Bind a hipStream_t (passed as void*; NULL = the null stream). */
dsmp_status dsmp_set_stream(dsmp_handle* h, void* stream);

/* Message of the last failed call on this handle ("" if none). */
const char* dsmp_last_error(const dsmp_handle* h);

/* ------------------------------------------------------------------ sampling
 * Nystrom node sampling (Sec. 2.1: a subset of s nodes drawn at random from
 * the domain; Algorithm 1, node-sampling step).  Uniform sampling without
 * replacement: candidate m gets the key
 *     SplitMix64 output number m+1 after seeding the state with `seed`
 * (Steele, Lea, Flood, OOPSLA 2014) and the s candidates with the smallest
 * keys are kept.  Keys are distinct, so the set is unique.
 *
 * idx_out : device int32 [s], receives the kept candidates in ascending order.
 * ws      : device workspace of at least dsmp_sample_workspace(M) bytes.
 * Errors  : INVALID_ARG if M < 0, s < 0, s > M, or a needed pointer is NULL.
 *           s == 0 enqueues nothing. */
dsmp_status dsmp_sample_workspace(int64_t M, size_t* bytes);
dsmp_status dsmp_sample_nodes(dsmp_handle* h, int64_t M, int64_t s, uint64_t seed,
                              int32_t* idx_out, void* ws, size_t ws_bytes);

/* Allocation-free variant of dsmp_sample_nodes, for callers that cannot
 * allocate or pass workspace (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation).  Same arguments and result,
 * without ws: the selection runs on a scratch array the library holds in
 * device memory, one per GPU for the life of the process (328 KB), sized for
 * at most 16,777,216 candidates; M beyond that gives UNSUPPORTED before
 * anything is enqueued.  Calls no allocating routine.  Every call on a GPU
 * uses that GPU's one array (its state and histogram are cleared by a kernel
 * at the start of each call), so calls that overlap on one GPU -- on two
 * streams, or from two threads -- race; serialise them. */
dsmp_status dsmp_sample_nodes_noalloc(dsmp_handle* h, int64_t M, int64_t s, uint64_t seed,
                                      int32_t* idx_out);

/* Gather rows: dst[i, :] = src[idx[i], :] for i < n.  Rows are row_bytes long
 * (a multiple of 4).  src: device [n_src_rows, row_bytes]; idx: device
 * int32 [n]; dst: device [n, row_bytes].  Indices out of [0, n_src_rows)
 * write a zero row.  Used to pull the sampled nodes' positions, attributes
 * and features out of the candidate arrays. */
dsmp_status dsmp_gather_rows(dsmp_handle* h, const void* src, int64_t n_src_rows,
                             int64_t row_bytes, const int32_t* idx, int64_t n, void* dst);

/* ------------------------------------------------------------- sub-domains
 * Sub-domain inference (Sec. 3, Methodology, testing procedure): the domain
 * is cut into smaller sub-domains, each with an overlap region; each is run
 * through the trained model as a graph of its own, and the outputs of its
 * own (interior) nodes are put back into the output over the whole domain.
 *
 * dsmp_subdomain_select picks the nodes of the box [lo, hi) (half-open in
 * every axis) with overlap l:
 *     owned   : lo[a] <= p[a] < hi[a] for every axis a
 *     overlap : not owned, and (lo[a] - l) <= p[a] < (hi[a] + l) for every a,
 *               the two bounds rounded to float32
 * pos     : device float32 [n, dim]; lo, hi: host float32 [dim]; overlap >= 0.
 * idx_out : device int32 [n] (capacity n); receives the owned nodes in
 *           ascending order at [0, *n_owned), then the overlap nodes in
 *           ascending order up to *n_total -- the layout the radius graph and
 *           the layer expect (destinations first).
 * ws      : device workspace of dsmp_subdomain_workspace(n) bytes.
 * SYNCHRONISES the stream; *n_owned and *n_total are host int64.
 * Errors  : INVALID_ARG for NULL pointers, n < 0 or overlap < 0;
 *           UNSUPPORTED for dim not 2 or 3; WORKSPACE_TOO_SMALL.
 * The kernels are timed in the DSMP_K_GATHER class. */
dsmp_status dsmp_subdomain_workspace(int64_t n, size_t* bytes);
dsmp_status dsmp_subdomain_select(dsmp_handle* h, const float* pos, int64_t n, int32_t dim,
                                  const float* lo, const float* hi, float overlap,
                                  int32_t* idx_out, void* ws, size_t ws_bytes,
                                  int64_t* n_owned, int64_t* n_total);

/* Scatter rows, the inverse of dsmp_gather_rows: dst[idx[i], :] = src[i, :]
 * for i < n (reassembly of a sub-domain's owned outputs).  src: device
 * [n, row_bytes]; idx: device int32 [n], distinct (two equal indices leave
 * either row); dst: device [n_dst_rows, row_bytes].  Indices outside
 * [0, n_dst_rows) are skipped.  row_bytes is a multiple of 4. */
dsmp_status dsmp_scatter_rows(dsmp_handle* h, const void* src, int64_t n, int64_t row_bytes,
                              const int32_t* idx, void* dst, int64_t n_dst_rows);

/* ------------------------------------------------------------- radius graph
 * Graph kernels of Sec. 2.1: every destination i in [0, n_dst) is joined to
 * every source j in [0, n_src), j != i, within radius r; when more than `cap`
 * sources qualify, `cap` of them are kept (Algorithm 1, edge-index creation
 * then edge sampling).  Sources are owned nodes first (the destinations)
 * then halo nodes of a sub-domain.
 *
 * The radius test is float32 without fused multiply-add, in this order:
 *     dx_a = p_j[a] - p_i[a];  d2 = ((dx_0*dx_0) + (dx_1*dx_1)) [+ (dx_2*dx_2)]
 *     keep iff d2 <= r*r      (r*r rounded to float32)
 * Cap modes: DSMP_CAP_KNN keeps the `cap` smallest (d2, j) pairs;
 * DSMP_CAP_RANDOM keeps the `cap` smallest (key, j) pairs where key is the
 * SplitMix64 output number i*n_src + j + 1 after seeding with `seed`, a
 * uniform random subset (the paper's edge sampling).
 *
 * Output (CSR by destination, deterministic): within each row the sources
 * are ascending.  dst[e] is the row of edge e.  csc_ptr/csc_eid group the
 * edges by source with ascending edge ids inside each group.
 */
enum { DSMP_CAP_KNN = 0, DSMP_CAP_RANDOM = 1 };

typedef struct dsmp_graph_query {
  const float* pos;   /* device float32 [n_src, dim], row-major */
  int64_t n_src;      /* >= n_dst */
  int64_t n_dst;      /* destinations are sources [0, n_dst) */
  int32_t dim;        /* 2 or 3 */
  float r;            /* radius, >= 0 */
  int32_t cap;        /* 0 = keep all, else the maximum edges per destination */
  int32_t cap_mode;   /* DSMP_CAP_KNN or DSMP_CAP_RANDOM */
  uint64_t seed;      /* used by DSMP_CAP_RANDOM */
} dsmp_graph_query;

typedef struct dsmp_graph {
  int64_t n_dst;
  int64_t n_src;
  int64_t n_edges;    /* E */
  int32_t* row_ptr;   /* device [n_dst+1] */
  int32_t* col;       /* device [E]  source of each edge */
  int32_t* dst;       /* device [E]  destination of each edge */
  int32_t* csc_ptr;   /* device [n_src+1] */
  int32_t* csc_eid;   /* device [E]  edge ids grouped by source */
} dsmp_graph;

/* Workspace bytes for count/build of this query (for a cap of 1..64 it
 * includes 8 * n_dst * cap bytes for the rows selected in one pass). */
dsmp_status dsmp_radius_graph_workspace(const dsmp_graph_query* q, size_t* bytes);

/* Count the edges.  SYNCHRONISES the stream; *n_edges (host) receives E.
 * UNSUPPORTED if a destination has more candidate sources than the per-row
 * limit (4096) or E exceeds 2^31-1. */
dsmp_status dsmp_radius_graph_count(dsmp_handle* h, const dsmp_graph_query* q, void* ws,
                                    size_t ws_bytes, int64_t* n_edges);

/* Build the graph into caller buffers (g->row_ptr ... g->csc_eid, sized for
 * `edge_capacity` edges).  SYNCHRONISES the stream once, after the row counts
 * (the host reads E), and writes g->n_dst, g->n_src and g->n_edges; the rows
 * and the transpose are queued on the stream after it.  If E > edge_capacity it returns
 * DSMP_CAPACITY with g->n_edges = E; then row_ptr is complete, and no edge
 * array has been written past edge_capacity. */
dsmp_status dsmp_radius_graph_build(dsmp_handle* h, const dsmp_graph_query* q, void* ws,
                                    size_t ws_bytes, int64_t edge_capacity, dsmp_graph* g);

/* --------------------------------------------------------------- NNConv layer
 * The edge-conditioned convolution of eq. (1) / eq. (ii) with the residual
 * hop update of Algorithm 1.  For edge e = (i <- j) with attributes x_e:
 *     z1 = ReLU(W1 x_e + b1),  z = ReLU(W2 z1 + b2)
 *     Theta_e[p][q] = (W3 z + b3)[p*d + q]            (never materialised)
 *     m_e[q] = sum_p Theta_e[p][q] * h_j[p]
 *     agg_i = mean of m_e over the edges of i (0 when i has none)
 *     y_i = agg_i + Wr h_i + br;   out_i = h_i + act(y_i)   (residual on)
 *                                  out_i = act(y_i)         (residual off)
 * Edge attributes: DSMP_ATTR_CONCAT  x_e = [p_i, p_j, s_i, s_j]  (de = 2*dim+2)
 *                  DSMP_ATTR_DIFF    x_e = v_i - v_j             (de = dim+1)
 * from node_attr rows v = (p, s) of dim+1 floats.
 *
 * dtype DSMP_BF16: h_in, W2, W3 and Wr take bfloat16 operands (the values in
 * the fp32 parameter arrays are rounded to nearest-even when packed) and the
 * products accumulate in float32; DSMP_F32 is float32 throughout.  Node
 * attributes, W1, biases, outputs and gradients are float32 in both.
 * Supported widths: d in {32, 64, 128}; h1, h2 in {32, 64, 128, 256};
 * dim in {2, 3}; other values give UNSUPPORTED.
 */
enum { DSMP_F32 = 0, DSMP_BF16 = 1 };
enum { DSMP_ACT_IDENTITY = 0, DSMP_ACT_RELU = 1 };
enum { DSMP_ATTR_CONCAT = 0, DSMP_ATTR_DIFF = 1 };
/* Backward flags: DSMP_GRAD_ACCUMULATE adds parameter gradients to the
 * caller's arrays (parameters shared by several layers or hops);
 * DSMP_GRAD_X_ACCUMULATE does the same for the input-side gradients that a
 * call documents as optional (a layer's dattr, a perceptron's grad_x). */
enum { DSMP_GRAD_ACCUMULATE = 1, DSMP_GRAD_X_ACCUMULATE = 2 };

typedef struct dsmp_layer_desc {
  int32_t dim;        /* spatial dimension D */
  int32_t d;          /* latent width */
  int32_t h1, h2;     /* kernel-MLP hidden widths */
  int32_t dtype;      /* DSMP_F32 or DSMP_BF16 */
  int32_t act;        /* DSMP_ACT_IDENTITY or DSMP_ACT_RELU */
  int32_t residual;   /* 0 or 1 */
  int32_t attr_mode;  /* DSMP_ATTR_CONCAT or DSMP_ATTR_DIFF */
} dsmp_layer_desc;

/* Parameters, device float32, torch Linear layout [out, in]:
 * W1 [h1, de], b1 [h1], W2 [h2, h1], b2 [h2], W3 [d*d, h2], b3 [d*d],
 * Wr [d, d], br [d]. */
typedef struct dsmp_layer_params {
  const float *W1, *b1, *W2, *b2, *W3, *b3, *Wr, *br;
} dsmp_layer_params;

/* Gradients, device float32, same layouts as the parameters.  dattr is
 * optional (NULL: not computed): for DSMP_ATTR_DIFF layers, device float32
 * [n_src, dim+1], the gradient with respect to the node attribute rows v
 * through the edge attributes x_e = v_i - v_j (row i gains the sum of W1^T da1
 * over its incoming edges, row j loses it over its outgoing ones; the step
 * that carries a hop's decoder outputs into the next hop's edge attributes,
 * eq. (iv) and Algorithm 1), overwritten, or added to when the backward's
 * flags have DSMP_GRAD_X_ACCUMULATE; UNSUPPORTED for DSMP_ATTR_CONCAT
 * layers. */
typedef struct dsmp_layer_grads {
  float *dW1, *db1, *dW2, *db2, *dW3, *db3, *dWr, *dbr;
  float* dattr;
} dsmp_layer_grads;

/* Bytes of the packed parameter buffer (the layouts the kernels read). */
dsmp_status dsmp_nnconv_packed_bytes(const dsmp_layer_desc* desc, size_t* bytes);

/* Pack parameters into `packed` (device, dsmp_nnconv_packed_bytes long,
 * 256-byte aligned).  Asynchronous; the parameters may be freed or changed
 * once the stream has passed this call. */
dsmp_status dsmp_nnconv_pack(dsmp_handle* h, const dsmp_layer_desc* desc,
                             const dsmp_layer_params* params, void* packed);

/* Byte sizes, for a graph with g->n_dst, g->n_src, g->n_edges set:
 *   saved : written by forward, read by backward (per layer);
 *   fwd_ws, bwd_ws : scratch of the forward and backward calls. */
dsmp_status dsmp_nnconv_workspace(const dsmp_layer_desc* desc, const dsmp_graph* g,
                                  size_t* saved_bytes, size_t* fwd_ws_bytes,
                                  size_t* bwd_ws_bytes);

/* Forward.  node_attr: device float32 [n_src, dim+1]; h_in: device
 * [n_src, d] of the layer dtype; h_out: device float32 [n_dst, d];
 * h_out_lp: NULL or device [n_dst, d] of the layer dtype (a copy of h_out
 * rounded to the layer dtype, e.g. the owned rows of the next layer's
 * input); saved / ws: device, sizes from dsmp_nnconv_workspace.  Inputs are
 * not modified; outputs are overwritten.  Uses g->row_ptr, g->col, g->dst. */
dsmp_status dsmp_nnconv_forward(dsmp_handle* h, const dsmp_layer_desc* desc, const void* packed,
                                const dsmp_graph* g, const float* node_attr, const void* h_in,
                                float* h_out, void* h_out_lp, void* saved, size_t saved_bytes,
                                void* ws, size_t ws_bytes);

/* Backward of the forward call that filled `saved`.  grad_out: device
 * float32 [n_dst, d].  grad_h: device float32 [n_src, d]; every row is
 * written (rows of sources with no edges get only the root and residual
 * terms, halo rows only their edge terms).  Parameter gradients go to
 * `grads` (every pointer non-NULL), overwritten, or added to when `flags`
 * has DSMP_GRAD_ACCUMULATE (layers sharing parameters).  Uses the whole
 * graph including csc_ptr / csc_eid. */
dsmp_status dsmp_nnconv_backward(dsmp_handle* h, const dsmp_layer_desc* desc, const void* packed,
                                 const dsmp_graph* g, const float* node_attr, const void* h_in,
                                 const void* saved, size_t saved_bytes, const float* grad_out,
                                 float* grad_h, const dsmp_layer_grads* grads, int32_t flags,
                                 void* ws, size_t ws_bytes);

/* ---------------------------------------------------- encoder and decoder
 * The node-wise networks of the hop loop (eq. (i) encoder N_e, eq. (iii)
 * decoder N_d; Algorithm 1, node encoding and decoding steps): a three-layer
 * perceptron applied to every row,
 *     y = W3 ReLU(W2 ReLU(W1 x + b1) + b2) + b3,
 * float32 throughout, parameters in the [out, in] layout of a linear layer:
 * W1 [d_hid, d_in], b1 [d_hid], W2 [d_hid, d_hid], b2 [d_hid],
 * W3 [d_out, d_hid], b3 [d_out].  Widths 1..256 (d_hid a multiple of 4);
 * others give UNSUPPORTED. */
typedef struct dsmp_mlp_desc {
  int32_t d_in, d_hid, d_out;
} dsmp_mlp_desc;

typedef struct dsmp_mlp_params {
  const float *W1, *b1, *W2, *b2, *W3, *b3;
} dsmp_mlp_params;

typedef struct dsmp_mlp_grads {
  float *dW1, *db1, *dW2, *db2, *dW3, *db3;
} dsmp_mlp_grads;

/* Byte sizes for n rows: saved (written by forward, read by backward) and
 * the backward workspace. */
dsmp_status dsmp_mlp_workspace(const dsmp_mlp_desc* desc, int64_t n, size_t* saved_bytes,
                               size_t* bwd_ws_bytes);

/* Forward on n rows.  x: device float32 [n, d_in]; y: device float32
 * [n, d_out], overwritten; y_bf16: NULL or device bfloat16 [n, d_out] (y
 * rounded to nearest-even, e.g. the feature input of a bf16 layer); saved:
 * device, dsmp_mlp_workspace long. */
dsmp_status dsmp_mlp_forward(dsmp_handle* h, const dsmp_mlp_desc* desc, const dsmp_mlp_params* p,
                             const float* x, int64_t n, float* y, void* y_bf16, void* saved,
                             size_t saved_bytes);

/* Backward of the forward that filled `saved`: gradients of sum(grad_y * y).
 * grad_x: NULL or device float32 [n, d_in], overwritten, or added to when
 * flags has DSMP_GRAD_X_ACCUMULATE.  Parameter gradients (every pointer
 * non-NULL) are overwritten, or added to with DSMP_GRAD_ACCUMULATE (one
 * network applied at several hops). */
dsmp_status dsmp_mlp_backward(dsmp_handle* h, const dsmp_mlp_desc* desc, const dsmp_mlp_params* p,
                              const float* x, int64_t n, const void* saved, size_t saved_bytes,
                              const float* grad_y, float* grad_x, const dsmp_mlp_grads* grads,
                              int32_t flags, void* ws, size_t ws_bytes);

/* ------------------------------------------------------------ loss
 * Mean squared error on the interior points (Algorithm 1, local loss): the
 * mean of (pred - target)^2 over the rows with mask[i] != 0 and all c
 * components.  pred, target: device float32 [n, c]; mask: device uint8 [n];
 * loss: device float32 scalar, overwritten (0 when no row is interior);
 * grad: NULL or device float32 [n, c], overwritten with d loss / d pred
 * (zero on the other rows).  The sums run in a fixed order. */
dsmp_status dsmp_masked_mse_workspace(int64_t n, size_t* bytes);
dsmp_status dsmp_masked_mse(dsmp_handle* h, const float* pred, const float* target, const uint8_t* mask,
                            int64_t n, int32_t c, float* loss, float* grad, void* ws, size_t ws_bytes);

/* How the layer evaluates the edge contraction.  DSMP_EDGE_PER_EDGE forms
 * each message m_e on MFMA (edge tiles against streamed W3 chunks) and sums
 * them per destination.  DSMP_EDGE_AGGREGATE uses the linearity of the mean:
 * the per-destination sums S_i = sum_e [z_e; 1] (x) h_j are formed first and
 * contracted with W3 and b3 in one GEMM (the feature gradient likewise over
 * the edges of each source, and dW3 from the same S_i); the result is the
 * same up to floating-point summation order.  DSMP_EDGE_AUTO (the default)
 * takes the aggregate form when the mean in-degree times d is at least 512.
 * The setting applies to later forward and backward calls on the handle; a
 * backward must run with the algorithm of its forward.  Workspace sizes
 * cover either algorithm. */
enum { DSMP_EDGE_AUTO = 0, DSMP_EDGE_PER_EDGE = 1, DSMP_EDGE_AGGREGATE = 2 };
dsmp_status dsmp_set_edge_algorithm(dsmp_handle* h, int32_t algorithm);

/* ------------------------------------------------------------ kernel timing
 * Opt-in timing of the library's kernels with HIP events, for benchmarks.
 * While enabled, every launch (or launch group) of a kernel class below is
 * bracketed by a pair of hipEvents recorded on the bound stream; the events
 * are created on first use and owned by the handle.  dsmp_profile_read
 * SYNCHRONISES on the outstanding events, adds their elapsed times to the
 * class totals and returns the total milliseconds and the number of
 * bracketed launches since the last reset.  Disabled (the default) the calls
 * record nothing. */
enum {
  DSMP_K_SAMPLE = 0,    /* dsmp_sample_nodes */
  DSMP_K_GATHER = 1,    /* dsmp_gather_rows */
  DSMP_K_GRAPH = 2,     /* dsmp_radius_graph_build (whole call) */
  DSMP_K_EDGE_FWD = 3,  /* forward edge contraction kernel */
  DSMP_K_NODE_FWD = 4,  /* forward node update kernel */
  DSMP_K_NODE_BWD = 5,  /* backward node, root and db3 kernels */
  DSMP_K_EDGE_DH = 6,   /* feature-gradient edge contraction kernel */
  DSMP_K_DH_FINAL = 7,  /* feature-gradient assembly kernel */
  DSMP_K_DZ = 8,        /* dz / da2 / da1 kernel (either form; with the terms of DSMP_K_DH_U at h = 256) */
  DSMP_K_DW3 = 9,       /* dW3 kernels (split over edges, or over S) */
  DSMP_K_DW2 = 10,      /* dW2 split-over-edges kernel */
  DSMP_K_DW1 = 11,      /* dW1 kernel */
  DSMP_K_REDUCE = 12,   /* fixed-order gradient reductions */
  DSMP_K_EDGE_MLP = 13, /* kernel-MLP edge kernel (aggregate form) */
  DSMP_K_OUTER_FWD = 14,/* per-destination sums S_i (aggregate form) */
  DSMP_K_GEMM_FWD = 15, /* W3 GEMM over S (aggregate form) */
  DSMP_K_OUTER_DH = 16, /* per-source sums T_j (aggregate form) */
  DSMP_K_GEMM_DH = 17,  /* W3 GEMM over T (aggregate form) */
  DSMP_K_U_GEMM = 18,   /* U = g W3 GEMM of the aggregate dz */
  DSMP_K_ATTR = 19,     /* edge-attribute gradient of a layer (dattr) */
  DSMP_K_MLP = 20,      /* encoder / decoder perceptrons, forward and backward */
  DSMP_K_LOSS = 21,     /* masked mean squared error */
  DSMP_K_DH_U = 22,     /* per-edge feature-gradient terms from U (aggregate form, bf16) */
  DSMP_K_DA1 = 23,      /* da1 from the stored da2 (aggregate form, bf16, h = 256) */
  DSMP_K_COUNT = 24
};
dsmp_status dsmp_profile_enable(dsmp_handle* h, int enable);
dsmp_status dsmp_profile_reset(dsmp_handle* h);
dsmp_status dsmp_profile_read(dsmp_handle* h, int kernel_class, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* DSMPNN_H */
