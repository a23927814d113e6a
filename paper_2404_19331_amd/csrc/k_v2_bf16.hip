// NHWC LDS-DMA kernel instances, element type bf16.
#define FCM_DT ::fcm::TBF16
#define FCM_TABLE_FN variants_v2_bf16
#include "k_v2.inc"
