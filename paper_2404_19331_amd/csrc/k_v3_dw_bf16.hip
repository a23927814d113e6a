#define FCM_DT TBF16
#define FCM_DT_NAME "bf16"
#define FCM_TABLE_FN variants_v3_dw_bf16
#define FCM_V3_TABLE FCM_V3_DW(3, 1, 4, 16), FCM_V3_DW(3, 1, 4, 32), FCM_V3_DW(3, 2, 4, 16), FCM_V3_DW(3, 2, 4, 32), FCM_V3_DW(5, 1, 4, 32), FCM_V3_DW(5, 2, 4, 32)
#include "k_v3.inc"
