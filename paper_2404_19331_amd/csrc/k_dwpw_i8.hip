// DW->PW and PW-only kernel instances, element type i8.
#define FCM_DT ::fcm::TI8
#define FCM_TABLE_FN variants_dwpw_i8
#include "k_dwpw.inc"
