// Instantiations of the 32x32x16 qlinear kernel (qmma_kernel.h) for 4-bit codes.
#include "qmma_kernel.h"

namespace subspec {

#define SUBSPEC_QMMA(G, MB, NB, PF) {MB, NB, PF, 4, G, qmma::k_qmma<4, G, MB, NB, PF>}

// Four row blocks (M = 65..128), the ring two chunks deep (two workgroups per CU) or
// four (one workgroup per CU, for launches split along a long K).
static const MmaVariant kVariants[] = {
    SUBSPEC_QMMA(128, 4, 1, 2), SUBSPEC_QMMA(128, 4, 1, 4), SUBSPEC_QMMA(64, 4, 1, 2), SUBSPEC_QMMA(64, 4, 1, 4),
};

const MmaVariant* qmma_variants_b4(int* n) {
  *n = static_cast<int>(sizeof(kVariants) / sizeof(kVariants[0]));
  return kVariants;
}

}  // namespace subspec
