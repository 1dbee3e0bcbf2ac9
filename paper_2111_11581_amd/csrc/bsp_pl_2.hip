// Instantiations of the identity-list pointwise kernel: bf16, stride 2.
#include "bsp_pl.h"

namespace bsp {
namespace pl {

pl_fn pick_2(int NSUB, int TM, bool map) { return pl_pick<2>(NSUB, TM, map); }

}  // namespace pl
}  // namespace bsp
