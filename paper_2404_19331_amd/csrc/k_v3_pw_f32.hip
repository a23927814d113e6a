#define FCM_DT TF32
#define FCM_DT_NAME "f32"
#define FCM_TABLE_FN variants_v3_pw_f32
#define FCM_V3_TABLE FCM_V3_PW(4, 4, 16), FCM_V3_PW(2, 8, 16), FCM_V3_PW(4, 4, 32)
#include "k_v3.inc"
