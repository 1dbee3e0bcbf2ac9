// Instantiations of the forward kernel: bf16, per-element gathers (any stride).
#include "bsp_fwd.h"

namespace bsp {
namespace fwd {

fwd_fn pick_b0(int TM, int TPG, int KS, bool map) { return pick_tm<uint16_t, 0, 2, 2>(TM, TPG, KS, map); }

}  // namespace fwd
}  // namespace bsp
