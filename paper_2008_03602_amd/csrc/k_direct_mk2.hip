// Instantiations of family 1 (DIRECT_F32) with MK = 2 output channels per thread.
#include "k_direct.inc.h"

namespace ct {
DirectFn pick_direct_mk2(int mw, int lds, int spec, int unr) { return pick_mw<2>(mw, lds, spec, unr); }
}  // namespace ct
