#define FCM_DT TBF16
#define FCM_DT_NAME "bf16"
#define FCM_TABLE_FN variants_v3_pw
#define FCM_V3_TABLE FCM_V3_PW(4, 4, 16), FCM_V3_PW(2, 8, 16), FCM_V3_PW(2, 16, 16), FCM_V3_PW2(2, 8, 16), FCM_V3_PW2(2, 16, 16), FCM_V3_PW(4, 4, 32), FCM_V3_PW(2, 8, 32)
#include "k_v3.inc"
