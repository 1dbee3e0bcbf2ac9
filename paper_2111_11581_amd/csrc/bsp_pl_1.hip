// Instantiations of the identity-list pointwise kernel: bf16, stride 1.
#include "bsp_pl.h"

namespace bsp {
namespace pl {

pl_fn pick_1(int NSUB, int TM, bool map) { return pl_pick<1>(NSUB, TM, map); }

}  // namespace pl
}  // namespace bsp
