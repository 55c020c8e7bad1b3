// Forward variants with FP8 (E4M3) P and V payloads (kernel in fwd_mxfp4.hpp):
// MXFP4 QK, P = E4M3(2^(y - E_B + 7)) with the Direct-P block exponent, MXFP8 V;
// online reference, noncausal and causal.
#include "fwd_mxfp4.hpp"

namespace fp4attn {
namespace directp_detail {

FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DEFINE, 0, kVarOnline | kPV8)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DEFINE, 0, kVarCausal | kPV8)

}  // namespace directp_detail
}  // namespace fp4attn
