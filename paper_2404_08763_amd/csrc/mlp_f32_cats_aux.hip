// Instantiations of the fused MLP kernel: f32 weights, cats aux variant.
#include "mlp_fused.hpp"

namespace cats {

hipError_t launch_fused_f32_cats_aux(int nch, int bt, const FusedArgs& a, int G, hipStream_t s) {
  return launch_fused_t<wf32, false, true>(nch, bt, a, G, s);
}

}  // namespace cats
