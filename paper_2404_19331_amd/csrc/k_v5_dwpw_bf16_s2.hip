#define FCM_DT TBF16
#define FCM_DT_NAME "bf16"
#define FCM_TABLE_FN variants_v5_dwpw_bf16_s2
#define FCM_V5_TABLE FCM_V5_DWPW(3, 2, 8, 14, 8, 1), FCM_V5_DWPW(3, 2, 4, 14, 8, 1), FCM_V5_DWPW(3, 2, 8, 14, 4, 1), FCM_V5_DWPW(3, 2, 7, 14, 4, 2), FCM_V5_DWPW(3, 2, 4, 14, 4, 4), FCM_V5_DWPW(3, 2, 7, 7, 4, 4), FCM_V5_DWPW(3, 2, 7, 7, 8, 2)
#include "k_v5.inc"
