// Instantiations of the pointwise kernel with gathered lists: bf16, stride 1.
#include "bsp_pl.h"

namespace bsp {
namespace pl {

pl_fn pick_g(int NSUB, int TM, int G) { return pl_pick_g(NSUB, TM, G); }

}  // namespace pl
}  // namespace bsp
