// DW->PW and PW-only kernel instances, element type bf16.
#define FCM_DT ::fcm::TBF16
#define FCM_TABLE_FN variants_dwpw_bf16
#include "k_dwpw.inc"
