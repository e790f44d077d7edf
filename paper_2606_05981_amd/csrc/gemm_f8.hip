// Instantiations of the projection GEMM for e4m3 weights (MODE_F8W), built
// as a translation unit of their own so that they compile in parallel with
// the fp16 / fp32 ones.
#include "gemm_kernel.h"

namespace mte {

hipError_t launch_mode_f8w(int epi, int tile, int splits, const GemmArgs &a, hipStream_t s) {
  return launch_mode<MODE_F8W>(epi, tile, splits, a, s);
}

}  // namespace mte
