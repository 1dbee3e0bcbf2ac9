// Instantiations of the forward kernel: bf16, stride-1 gathers, no step split.
#include "bsp_fwd.h"

namespace bsp {
namespace fwd {

fwd_fn pick_b1_k1(int TM, int TPG, int KS, bool map) { return pick_tm<uint16_t, 1, 2, 4>(TM, TPG, KS, map); }

}  // namespace fwd
}  // namespace bsp
