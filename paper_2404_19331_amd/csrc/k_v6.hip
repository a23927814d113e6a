// Instances of the whole-module fp32 kernels for small batches (fcm_kernels_v6.h):
// (module, k, stride, tile rows, tile columns).
#include "fcm_kernels_v6.h"

namespace fcm {

#define FCM_V6(FAM, MODE, K, S, TH, TW, NAME)                                                                 \
  Variant{FAM, DT_F32, K, S, TH * TW, 0, 0, 0, 0, &launch_small6<MODE, K, S, TH, TW>,                       \
          NAME "<f32," #K "," #S "," #TH "x" #TW ">", TH, TW, 6, 0, 1, 1}
#define FCM_V6_DWPW(K, S, TH, TW) FCM_V6(FAM_DWPW, M6_DWPW, K, S, TH, TW, "k_dwpw6")
#define FCM_V6_PWDW(K, S, TH, TW) FCM_V6(FAM_PWDW, M6_PWDW, K, S, TH, TW, "k_pwdw6")
#define FCM_V6_PWDWPW(K, S, TH, TW) FCM_V6(FAM_PWDWPW, M6_PWDWPW, K, S, TH, TW, "k_pwdwpw6")

static const Variant kTable[] = {
    FCM_V6_DWPW(3, 1, 4, 4),     FCM_V6_DWPW(3, 1, 4, 8),     FCM_V6_DWPW(3, 1, 8, 8),   FCM_V6_DWPW(3, 1, 2, 8),
    FCM_V6_DWPW(3, 2, 4, 4),     FCM_V6_DWPW(3, 2, 4, 8),     FCM_V6_DWPW(5, 1, 4, 4),   FCM_V6_DWPW(5, 2, 4, 4),
    FCM_V6_PWDW(3, 1, 4, 4),     FCM_V6_PWDW(3, 1, 4, 8),     FCM_V6_PWDW(3, 2, 4, 4),   FCM_V6_PWDWPW(3, 1, 4, 4),
    FCM_V6_PWDWPW(3, 1, 4, 8),   FCM_V6_PWDWPW(3, 1, 2, 8),   FCM_V6_PWDWPW(3, 1, 2, 4), FCM_V6_PWDWPW(3, 2, 4, 4),
    FCM_V6_PWDWPW(5, 1, 4, 4)};

const Variant* variants_v6_f32(int* count) {
  *count = (int)(sizeof(kTable) / sizeof(kTable[0]));
  return kTable;
}

}  // namespace fcm
