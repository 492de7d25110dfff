// ProxyFormer layer backward (placeholder until the backward kernels land).
#include "common.hpp"
#include "layer.hpp"

namespace pf {

size_t layer_backward_gemm_ws(const LayerDims&) { return 0; }

template <typename T>
hipError_t layer_backward_run(const LayerDims&, const pf_layer_config*, const pf_layer_weights*, const void*,
                              const void*, const char*, const void*, const void*, void*, void*,
                              const pf_layer_grads*, char*, hipStream_t) {
  return hipErrorNotSupported;
}

template hipError_t layer_backward_run<bf16>(const LayerDims&, const pf_layer_config*, const pf_layer_weights*,
                                             const void*, const void*, const char*, const void*, const void*, void*,
                                             void*, const pf_layer_grads*, char*, hipStream_t);
template hipError_t layer_backward_run<float>(const LayerDims&, const pf_layer_config*, const pf_layer_weights*,
                                              const void*, const void*, const char*, const void*, const void*, void*,
                                              void*, const pf_layer_grads*, char*, hipStream_t);
}  // namespace pf
