// Direct-P forward variants with native-exponential pair mixing, 1, 2, 4 of the
// 16 pairs of each 32-key block (kernel in fwd_mxfp4.hpp).
#include "fwd_mxfp4.hpp"

namespace fp4attn {
namespace directp_detail {

FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DEFINE, 1, kVarOnline)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DEFINE, 2, kVarOnline)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DEFINE, 4, kVarOnline)

}  // namespace directp_detail
}  // namespace fp4attn
