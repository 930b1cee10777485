// Attention over block-scaled integer caches (App. C, quantized KV caches) on the bf16
// path: the kernels of attention_kernels.hpp instantiated for int8 and int4 keys and
// values. Kept in a translation unit of its own so that it compiles in parallel with
// the plain kernels.
#include "attention_kernels.hpp"

namespace pkv {

hipError_t run_attention_mx(const AttnShape& s, const AttnPlan& pl, AttnParams& p, int bits,
                            bool gather, bool psplit, hipStream_t st) {
  if (bits == 8)
    return s.dh == 128 ? run_attention<128, 8>(s, pl, p, gather, psplit, st)
                       : run_attention<64, 8>(s, pl, p, gather, psplit, st);
  if (bits == 4)
    return s.dh == 128 ? run_attention<128, 4>(s, pl, p, gather, psplit, st)
                       : run_attention<64, 4>(s, pl, p, gather, psplit, st);
  return hipErrorInvalidValue;
}

}  // namespace pkv
