// Instantiations of the fused MLP kernel: fp32 weights, top-k variant (v and
// the per-row cutoffs precomputed).
#include "mlp_fused.hpp"

namespace cats {

hipError_t launch_fused_f32_topk(int nch, int bt, bool aux, const FusedArgs& a, int G, hipStream_t s) {
  return aux ? launch_fused_t<wf32, false, true, true>(nch, bt, a, G, s)
             : launch_fused_t<wf32, false, false, true>(nch, bt, a, G, s);
}

}  // namespace cats
