// PW->DW->PW and PW->PW kernel instances, all element types.
// (QMAX haloed positions, intermediate chunk MBMAX, output block OMAX, PMAX output pixels)
#include "fcm_kernels.h"

namespace fcm {

#define FCM_PDP(DT, K, S, OM, WM2)                                                                     \
  {FAM_PWDWPW, dtype_id<DT>(), K, S, 64, 128, OM, 64, 4, &launch_pwdwpw<DT, K, S, 128, 64, 1, OM, 64, WM2, 4, true>, \
   "k_pwdwpw<" #DT "," #K "," #S "," #OM ">"}
#define FCM_PDP_KS(DT, K, S) FCM_PDP(DT, K, S, 32, 1), FCM_PDP(DT, K, S, 128, 2)
#define FCM_PDP_DT(DT) FCM_PDP_KS(DT, 3, 1), FCM_PDP_KS(DT, 3, 2), FCM_PDP_KS(DT, 5, 1), FCM_PDP_KS(DT, 5, 2)
// PW -> PW: window = tile (64 positions), the depthwise stage compiled out
#define FCM_PP(DT, OM, WM2)                                                                          \
  {FAM_PWPW, dtype_id<DT>(), 1, 1, 64, 64, OM, 64, 4, &launch_pwdwpw<DT, 1, 1, 64, 64, 1, OM, 64, WM2, 4, false>, \
   "k_pwpw<" #DT "," #OM ">"}
#define FCM_PP_DT(DT) FCM_PP(DT, 32, 1), FCM_PP(DT, 128, 2)

static const Variant kTable[] = {FCM_PDP_DT(TF32), FCM_PDP_DT(TBF16), FCM_PDP_DT(TI8),
                                 FCM_PP_DT(TF32), FCM_PP_DT(TBF16), FCM_PP_DT(TI8)};

const Variant* variants_pwdwpw(int* count) {
  *count = (int)(sizeof(kTable) / sizeof(kTable[0]));
  return kTable;
}

}  // namespace fcm
