// Direct-P forward variants with the sampled QK guard of Alg. 3 (kernel in
// fwd_mxfp4.hpp), for the all-affine map, the quarter of native-exponential
// pairs and the exp2-only route.
#include "fwd_mxfp4.hpp"

namespace fp4attn {
namespace directp_detail {

FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DEFINE, 0, kVarGuard)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DEFINE, 4, kVarGuard)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DEFINE, 16, kVarGuard)

}  // namespace directp_detail
}  // namespace fp4attn
