// Instantiations of the pointwise kernel: fp32, stride 1.
#include "bsp_pw.h"

namespace bsp {
namespace pw {

pw_fn pick_f(int TM, int TPG, int KS, bool map) { return pw_pick_tm<float, 1, 2 | 4 | 16, 2>(TM, TPG, KS, map); }

}  // namespace pw
}  // namespace bsp
