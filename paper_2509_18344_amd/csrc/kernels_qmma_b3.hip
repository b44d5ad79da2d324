// Instantiations of the 32x32x16 qlinear kernel (qmma_kernel.h) for 3-bit codes.
#include "qmma_kernel.h"

namespace subspec {

#define SUBSPEC_QMMA(G, MB, NB, PF, W) {MB, NB, PF, W, 1, 3, G, qmma::k_qmma<3, G, MB, NB, PF, W, 1>}
#define SUBSPEC_QMMA_TEAMS(G, MB) {MB, 1, 2, 8, 2, 3, G, qmma::k_qmma<3, G, MB, 1, 2, 8, 2>}

// Four row blocks (M = 65..128): four wavefronts with the ring two chunks deep (two
// workgroups per CU) or four (one workgroup per CU); eight wavefronts (256 columns, one
// workgroup per CU) with the ring four chunks deep (not with groups of 64, where that
// build spills registers).
// Two row blocks (M = 33..64): eight wavefronts (256 columns) with the ring four chunks
// deep.  Two teams of four wavefronts, each with a two-chunk ring, on long-K launches
// from M = 33 (64-row tiles) and above M = 64 (128-row tiles).
static const MmaVariant kVariants[] = {
    SUBSPEC_QMMA(128, 4, 1, 2, 4), SUBSPEC_QMMA(128, 4, 1, 4, 4), SUBSPEC_QMMA(128, 4, 1, 4, 8),
    SUBSPEC_QMMA(64, 4, 1, 2, 4),  SUBSPEC_QMMA(64, 4, 1, 4, 4),
    SUBSPEC_QMMA(128, 2, 1, 4, 8), SUBSPEC_QMMA(64, 2, 1, 4, 8),
    SUBSPEC_QMMA_TEAMS(128, 4), SUBSPEC_QMMA_TEAMS(64, 4),
    SUBSPEC_QMMA_TEAMS(128, 2), SUBSPEC_QMMA_TEAMS(64, 2),
};

const MmaVariant* qmma_variants_b3(int* n) {
  *n = static_cast<int>(sizeof(kVariants) / sizeof(kVariants[0]));
  return kVariants;
}

}  // namespace subspec
