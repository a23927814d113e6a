#define FCM_DT TF32
#define FCM_DT_NAME "f32"
#define FCM_TABLE_FN variants_v4_pwpw_f32
#include "k_v4.inc"
