// Instantiations of the forward kernel: fp32.
#include "bsp_fwd.h"

namespace bsp {
namespace fwd {

fwd_fn pick_f(int mode, int TM, int TPG, int KS, bool map) {
    return mode == 1 ? pick_tm<float, 1, 2, 2>(TM, TPG, KS, map) : pick_tm<float, 0, 2, 2>(TM, TPG, KS, map);
}

}  // namespace fwd
}  // namespace bsp
