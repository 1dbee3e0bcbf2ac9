// Instantiations of the forward kernel: bf16, stride-1 gathers, steps split over 2 or 4 waves.
#include "bsp_fwd.h"

namespace bsp {
namespace fwd {

fwd_fn pick_b1_k24(int TM, int TPG, int KS, bool map) { return pick_tm<uint16_t, 1, 4 | 16, 4>(TM, TPG, KS, map); }

}  // namespace fwd
}  // namespace bsp
