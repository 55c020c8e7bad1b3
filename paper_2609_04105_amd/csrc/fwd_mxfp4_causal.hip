// Causal Direct-P forward variants (kernel in fwd_mxfp4.hpp): the all-affine
// map, the quarter of native-exponential pairs and the exp2-only route.
#include "fwd_mxfp4.hpp"

namespace fp4attn {
namespace directp_detail {

FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DEFINE, 0, kVarCausal)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DEFINE, 4, kVarCausal)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DEFINE, 16, kVarCausal)

}  // namespace directp_detail
}  // namespace fp4attn
