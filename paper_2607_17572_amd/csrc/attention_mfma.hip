// MFMA (bf16) flash attention for head dim 128 on gfx950.  Placeholder until
// the MFMA kernels land: returns -1 so the caller takes the VALU kernels.
#include "attention.h"

namespace jg {
int attention_fwd_mfma(const AttnFwd&, hipStream_t) { return -1; }
int attention_bwd_mfma(const AttnBwd&, hipStream_t) { return -1; }
}  // namespace jg
