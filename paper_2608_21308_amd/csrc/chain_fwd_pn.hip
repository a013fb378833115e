// The forward chain kernels with the post-chunk normalisation of the fast
// weights: the same source, instantiated in a translation unit of its own.
#define E2TTT_CHAIN_PN 1
#include "chain_fwd.hip"
