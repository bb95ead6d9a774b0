// Decode attention over caches with on-demand sparse pages: the kernel of
// attention_mfma.hip instantiated for them in a translation unit of its own.
#define OAKEN_ATTN_PAGED_TU 1
#include "attention_mfma.hip"
