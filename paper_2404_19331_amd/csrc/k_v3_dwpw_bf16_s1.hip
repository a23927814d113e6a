#define FCM_DT TBF16
#define FCM_DT_NAME "bf16"
#define FCM_TABLE_FN variants_v3_dwpw_bf16_s1
#define FCM_V3_TABLE FCM_V3_DWPW(3, 1, 4, 4, 16), FCM_V3_DWPW(3, 1, 2, 8, 16), FCM_V3_DWPW(3, 1, 1, 16, 16), FCM_V3_DWPW2(3, 1, 1, 16, 16), FCM_V3_DWPW2(3, 1, 2, 8, 16), FCM_V3_DWPW2(3, 1, 4, 4, 16), FCM_V3_DWPW(3, 1, 4, 4, 32), FCM_V3_DWPW(3, 1, 2, 8, 32), FCM_V3_DWPW(5, 1, 4, 4, 32), FCM_V3_DWPW(5, 1, 2, 8, 32)
#include "k_v3.inc"
