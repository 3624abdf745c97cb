// Instantiations of family 4 (IGEMM_F32): 16x16 fp32 MFMA shape, TM = 2.
#include "k_igemm_f32.inc.h"

namespace ct {
IgF32Fn igf32_pick_mf16_tm2(int tn, int stages, int spec) { return igf32_pick_tn<16, 2>(tn, stages, spec); }
}  // namespace ct
