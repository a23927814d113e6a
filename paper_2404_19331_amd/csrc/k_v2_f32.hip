// NHWC LDS-DMA kernel instances, element type f32.
#define FCM_DT ::fcm::TF32
#define FCM_TABLE_FN variants_v2_f32
#include "k_v2.inc"
