#define FCM_DT TBF16
#define FCM_DT_NAME "bf16"
#define FCM_TABLE_FN variants_v4_pwpw_bf16
#include "k_v4.inc"
