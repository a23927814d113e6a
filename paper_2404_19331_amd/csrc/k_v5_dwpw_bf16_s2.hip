#define FCM_DT TBF16
#define FCM_DT_NAME "bf16"
#define FCM_TABLE_FN variants_v5_dwpw_bf16_s2
#define FCM_V5_TABLE FCM_V5_DWPW(3, 2, 2, 4, 1), FCM_V5_DWPW(3, 2, 2, 8, 1), FCM_V5_DWPW(3, 2, 4, 4, 2), FCM_V5_DWPW(3, 2, 4, 8, 2), FCM_V5_DWPW(3, 2, 4, 4, 4), FCM_V5_DWPW(3, 2, 8, 4, 4), FCM_V5_DWPW(3, 2, 4, 8, 4)
#include "k_v5.inc"
