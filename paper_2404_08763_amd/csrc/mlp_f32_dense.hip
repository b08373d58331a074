// Instantiations of the fused MLP kernel: f32 weights, dense variant.
#include "mlp_fused.hpp"

namespace cats {

hipError_t launch_fused_f32_dense(int nch, int bt, const FusedArgs& a, int G, hipStream_t s) {
  return launch_fused_t<wf32, true, false>(nch, bt, a, G, s);
}

}  // namespace cats
