// Instantiations of the pointwise kernel: bf16, stride 1.
#include "bsp_pw.h"

namespace bsp {
namespace pw {

pw_fn pick_b1(int TM, int TPG, int KS, bool map) { return pw_pick_tm<uint16_t, 1, 2 | 4 | 16, 4>(TM, TPG, KS, map); }

}  // namespace pw
}  // namespace bsp
