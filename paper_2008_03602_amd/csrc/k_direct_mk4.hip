// Instantiations of family 1 (DIRECT_F32) with MK = 4 output channels per thread.
#include "k_direct.inc.h"

namespace ct {
DirectFn pick_direct_mk4(int mw, int lds, int spec, int unr) { return pick_mw<4>(mw, lds, spec, unr); }
}  // namespace ct
