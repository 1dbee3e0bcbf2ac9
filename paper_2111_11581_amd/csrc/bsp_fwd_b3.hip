// Instantiations of the forward kernel: bf16, stride-1 gathers at any element.
#include "bsp_fwd.h"

namespace bsp {
namespace fwd {

fwd_fn pick_b3(int TM, int TPG, int KS, bool map) { return pick_tm<uint16_t, 3, 2 | 4 | 16, 4>(TM, TPG, KS, map); }

}  // namespace fwd
}  // namespace bsp
