#define FCM_DT TI8
#define FCM_DT_NAME "i8"
#define FCM_TABLE_FN variants_v4_pwpw_i8
#include "k_v4.inc"
