// Instances of the deep DW->PW kernels (fcm_kernels_v7.h): (stride, tile rows, tile
// columns, output tiles per wave: the channel block is 64 x that, 32-channel chunks per
// item).
#include "fcm_kernels_v7.h"

namespace fcm {

#define FCM_V7(S, TH, TW, CTW, KC, SUFFIX)                                                                   \
  Variant{FAM_DWPW, DT_BF16, 3, S, TH * TW, 0, 64 * CTW, 0, 0, &launch_deep7<S, TH, TW, CTW, KC>,              \
          "k_dwpw7<bf16,3," #S "," #TH "x" #TW ",ct" #CTW SUFFIX ">", TH, TW, 7, 0, 2, 4, KC}

static const Variant kTable[] = {FCM_V7(1, 7, 7, 4, 1, ""),     FCM_V7(1, 4, 14, 4, 1, ""), FCM_V7(1, 8, 8, 4, 1, ""),
                                 FCM_V7(1, 7, 7, 2, 1, ""),     FCM_V7(1, 4, 14, 2, 1, ""), FCM_V7(2, 7, 7, 4, 1, ""),
                                 FCM_V7(2, 4, 14, 4, 1, ""),    FCM_V7(2, 7, 7, 2, 1, ""),  FCM_V7(1, 7, 7, 4, 2, ",k2"),
                                 FCM_V7(1, 7, 7, 2, 2, ",k2"), FCM_V7(2, 7, 7, 4, 2, ",k2"), FCM_V7(2, 7, 7, 2, 2, ",k2"),
                                 FCM_V7(1, 4, 14, 4, 2, ",k2")};

const Variant* variants_v7_bf16(int* count) {
  *count = (int)(sizeof(kTable) / sizeof(kTable[0]));
  return kTable;
}

}  // namespace fcm
