// Instantiations of the fused MLP kernel: bf16 weights, top-k variant (v and
// the per-row cutoffs precomputed).
#include "mlp_fused.hpp"

namespace cats {

hipError_t launch_fused_bf16_topk(int nch, int bt, bool aux, const FusedArgs& a, int G, hipStream_t s) {
  return aux ? launch_fused_t<wbf16, false, true, true>(nch, bt, a, G, s)
             : launch_fused_t<wbf16, false, false, true>(nch, bt, a, G, s);
}

}  // namespace cats
