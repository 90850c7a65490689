// NNConv layer backward (placeholder until the backward kernels land).
#include "nnconv.hpp"

namespace dsmp {
struct SavedLayout { size_t y, zE, z1E, total; };
SavedLayout saved_layout(const dsmp_layer_desc& d, int64_t n_dst, int64_t E);
size_t fwd_ws_bytes(const dsmp_layer_desc& d, int64_t n_dst, int64_t E);
dsmp_status check_layer_desc(dsmp_handle* h, const dsmp_layer_desc* d);
}
using namespace dsmp;

extern "C" dsmp_status dsmp_nnconv_workspace(const dsmp_layer_desc* desc, const dsmp_graph* g,
                                             size_t* saved_bytes, size_t* fwd_ws, size_t* bwd_ws) {
  if (!desc || !g || !saved_bytes || !fwd_ws || !bwd_ws) return DSMP_INVALID_ARG;
  dsmp_status st = check_layer_desc(nullptr, desc);
  if (st != DSMP_OK) return st;
  *saved_bytes = saved_layout(*desc, g->n_dst, g->n_edges).total;
  *fwd_ws = fwd_ws_bytes(*desc, g->n_dst, g->n_edges);
  *bwd_ws = 256;
  return DSMP_OK;
}

extern "C" dsmp_status dsmp_nnconv_backward(dsmp_handle* h, const dsmp_layer_desc*, const void*,
                                            const dsmp_graph*, const float*, const void*, const void*,
                                            size_t, const float*, float*, const dsmp_layer_grads*,
                                            int32_t, void*, size_t) {
  return fail(h, DSMP_UNSUPPORTED, "backward not built yet");
}
