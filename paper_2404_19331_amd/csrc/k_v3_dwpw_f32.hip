#define FCM_DT TF32
#define FCM_DT_NAME "f32"
#define FCM_TABLE_FN variants_v3_dwpw_f32
#define FCM_V3_TABLE FCM_V3_DWPW(3, 1, 4, 4, 16), FCM_V3_DWPW(3, 1, 2, 8, 32), FCM_V3_DWPW(3, 2, 4, 4, 16), FCM_V3_DWPW(3, 2, 2, 8, 32), FCM_V3_DWPW(5, 1, 4, 4, 32), FCM_V3_DWPW(5, 2, 4, 4, 32)
#include "k_v3.inc"
