// bf16 MFMA flash attention for gfx950 (placeholder until the MFMA tiling lands).
#include "common.h"
#include "kernels.h"

bool attention_mfma_fwd_try(const AttnArgs&, hipStream_t) { return false; }
bool attention_mfma_bwd_try(const AttnArgs&, hipStream_t) { return false; }
