#define FCM_DT TI8
#define FCM_DT_NAME "i8"
#define FCM_TABLE_FN variants_v3_pw_i8
#define FCM_V3_TABLE FCM_V3_PW(4, 4, 16), FCM_V3_PW(2, 8, 16), FCM_V3_PW(4, 4, 32)
#include "k_v3.inc"
