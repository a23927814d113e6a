#define FCM_DT TBF16
#define FCM_DT_NAME "bf16"
#define FCM_TABLE_FN variants_v5_pwdw_bf16
#define FCM_V5_TABLE FCM_V5_PW(8, 16, 4, 1), FCM_V5_PW(8, 16, 8, 1), FCM_V5_DW(3, 1, 8, 16), FCM_V5_DW(3, 2, 8, 8)
#include "k_v5.inc"
