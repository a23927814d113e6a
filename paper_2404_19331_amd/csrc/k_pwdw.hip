// PW->DW and DW-only kernel instances, all element types.
#include "fcm_kernels.h"

namespace fcm {

#define FCM_PWDW(DT, K, S, QM, MM)                                                                      \
  {FAM_PWDW, dtype_id<DT>(), K, S, 0, QM, MM, 0, 4, &launch_pwdw<DT, K, S, true, QM, MM, 1, 4>,          \
   "k_pwdw<" #DT "," #K "," #S "," #QM "," #MM ">"}
#define FCM_DWONLY(DT, K, S)                                                                            \
  {FAM_DW, dtype_id<DT>(), K, S, 0, 0, 128, 0, 4, &launch_pwdw<DT, K, S, false, 64, 64, 1, 4>,           \
   "k_dw<" #DT "," #K "," #S ">"}
#define FCM_PWDW_KS(DT, K, S) FCM_PWDW(DT, K, S, 128, 64), FCM_PWDW(DT, K, S, 320, 64), FCM_DWONLY(DT, K, S)
#define FCM_PWDW_DT(DT) FCM_PWDW_KS(DT, 3, 1), FCM_PWDW_KS(DT, 3, 2), FCM_PWDW_KS(DT, 5, 1), FCM_PWDW_KS(DT, 5, 2)

static const Variant kTable[] = {FCM_PWDW_DT(TF32), FCM_PWDW_DT(TBF16), FCM_PWDW_DT(TI8)};

const Variant* variants_pwdw(int* count) {
  *count = (int)(sizeof(kTable) / sizeof(kTable[0]));
  return kTable;
}

}  // namespace fcm
