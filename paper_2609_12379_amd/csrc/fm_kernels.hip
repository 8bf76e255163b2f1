// Instantiates the step kernel for one batch specialisation FM_B (compiled once per value
// of FM_B in {1, 2, 4, 8}, so the builds run in parallel). Kernels are specialised on the
// batch, head_dim (64, 128) and the GQA group size (rounded up to 1, 2, 4, 8), so each
// carries only the code its model runs.
#include "fm_kernel.h"

#ifndef FM_B
#error "compile with -DFM_B=<1|2|4|8>"
#endif
#define FM_CAT2(a, b) a##b
#define FM_CAT(a, b) FM_CAT2(a, b)

namespace fm {
namespace dev {

#ifdef FM_STUB
// Development builds may leave a batch specialisation out; fm_create then reports it as
// unsupported.
const void* FM_CAT(kernel_for_b, FM_B)(int, int) { return nullptr; }
#else
template <int GT>
static const void* pick(int d) {
  return d == 64 ? (const void*)&step_kernel<FM_B, 64, GT> : (const void*)&step_kernel<FM_B, 128, GT>;
}

const void* FM_CAT(kernel_for_b, FM_B)(int d, int G) {
  switch (G) {
    case 1: return pick<1>(d);
    case 2: return pick<2>(d);
    case 3: case 4: return pick<4>(d);
    default: return pick<8>(d);
  }
}
#endif

}  // namespace dev
}  // namespace fm
