#define FCM_DT TBF16
#define FCM_DT_NAME "bf16"
#define FCM_TABLE_FN variants_v5_pwdw_bf16
#define FCM_V5_TABLE FCM_V5_PW(2, 4, 1), FCM_V5_PW(2, 8, 1), FCM_V5_PW(4, 4, 2), FCM_V5_PW(4, 8, 2), FCM_V5_PW(4, 4, 4), FCM_V5_PW(8, 4, 4), FCM_V5_DW(3, 1, 2), FCM_V5_DW(3, 2, 2), FCM_V5_DW(3, 1, 1), FCM_V5_DW(3, 2, 1)
#include "k_v5.inc"
