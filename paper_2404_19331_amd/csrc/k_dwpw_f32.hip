// DW->PW and PW-only kernel instances, element type f32.
#define FCM_DT ::fcm::TF32
#define FCM_TABLE_FN variants_dwpw_f32
#include "k_dwpw.inc"
