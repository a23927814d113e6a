// NHWC LDS-DMA kernel instances, element type i8.
#define FCM_DT ::fcm::TI8
#define FCM_TABLE_FN variants_v2_i8
#include "k_v2.inc"
