/*
 * fcm.h -- Fused Convolutional Modules (FCMs) for AMD Instinct MI355X (gfx950).
 *
 * C ABI of libfcm.so. Implements the fused depthwise (DW) / pointwise (PW) convolution
 * kernels of Qararyah et al., "Fusing Depthwise and Pointwise Convolutions for
 * Efficient Inference on GPUs" (arXiv 2404.19331), and the FusePlanner cost model that
 * chooses their tiling.
 *
 *   fcm_dw_pw     DW -> PW in one kernel (Sec. III-A "DWPW"; the depthwise separable
 *                 convolution of Sec. II-B). The DW output tile never leaves the chip.
 *   fcm_pw_dw     PW -> DW in one kernel (Sec. III-A "PWDW" / "PWDW_R"): the PW output is
 *                 recomputed on the DW halo of each spatial tile (Sec. II-D), or computed
 *                 once when a tile spans the whole plane.
 *   fcm_pw_dw_pw  PW -> DW -> PW in one kernel (the inverted-residual block of Sec. II-B,
 *                 three layers fused; the paper's modules fuse two).
 *   fcm_pw_pw     PW -> PW in one kernel (Sec. III-A "PwPw", two pointwise layers; the
 *                 first layer's output tile stays on chip, chunk by chunk).
 *   fcm_dw, fcm_pw  single layers ("layer-by-layer", LBL, Sec. II-D and V-C): the
 *                 unfused comparison, built from the same tiles and dataflow.
 *   fcm_plan      FusePlanner (Sec. IV): global-memory-access estimates of the LBL and
 *                 fused kernels (Eq. 1-4) and the tiling that minimises them.
 *   fcm_chain_plan, fcm_chain_run  FusePlanner over a sequence of DW/PW layers: which
 *                 adjacent layers to fuse into which module, then the chain's launches.
 *   fcm_fold_batchnorm  folds an inference batch normalisation into a float convolution.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  * Tensors are caller-owned DEVICE pointers (e.g. PyTorch tensors). Every launch is
 *    asynchronous on `stream` (a hipStream_t; NULL = the null stream); the library never
 *    allocates, frees or synchronises. Plans that split a work tile's channel chunks over
 *    several workgroups keep partial sums in a caller-provided device workspace
 *    (fcm_workspace_bytes, fcm_dw_pw_ws, fcm_pw_ws); the entry points without a workspace
 *    argument plan without splits and refuse a split plan with FCM_EINVAL. Calls that
 *    share one workspace must not overlap (e.g. on two streams).
 *  * Activations: x is [n, c, h, w] (FCM_NCHW) or [n, h, w, c] (FCM_NHWC), dense,
 *    row-major. The output uses the same layout.
 *  * Weights are canonical regardless of layout: depthwise [c][k][k] (PyTorch
 *    [c, 1, k, k]); pointwise [c_out][c_in] (PyTorch [c_out, c_in, 1, 1]).
 *  * Element types: FCM_F32 float; FCM_BF16 bfloat16 (raw 16-bit patterns; computed with
 *    fp32 accumulation, each stage's result rounded to bfloat16, nearest-even);
 *    FCM_I8 int8 (int32 accumulation, each stage requantised to int8 by
 *    desc->rq[stage], Sec. III-B).
 *  * Biases (folded normalisation, Sec. III-A "convolution-normalisation-activation")
 *    may be NULL (= zero): float for F32/BF16, int32 for I8.
 *  * Depthwise geometry: square k x k, stride `stride`, symmetric zero padding `pad`,
 *    channel multiplier 1; output h_o = (h + 2*pad - k)/stride + 1 (same for w).
 *  * Each conv stage computes conv -> +bias -> activation -> cast. act[i]/rq[i] belong to
 *    the i-th convolution in execution order.
 *  * Pointers must be aligned to their element size; 16-byte aligned tensors with
 *    16-byte multiple channel rows take the vector path (same results either way).
 *  * Errors are returned synchronously as fcm_status; fcm_last_error() gives a
 *    thread-local message. No exception crosses the ABI. Thread-safe.
 */
#ifndef FCM_H_
#define FCM_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* The largest workspace a split plan of the persistent DW->PW and PW kernels may need
 * (its partial sums); the planner does not split where they would exceed it. */
#define FCM_SPLIT_WORKSPACE_BYTES (64u << 20)

typedef enum {
  FCM_OK = 0,
  FCM_EINVAL = 1,        /* NULL tensor, non-positive size, bad geometry or requant  */
  FCM_EUNSUPPORTED = 2,  /* valid but not built: k not in {3,5}, stride not in {1,2},
                            plan that no compiled kernel implements,
                            tile that does not fit in LDS                              */
  FCM_EDEVICE = 3        /* HIP reported an error at launch                          */
} fcm_status;

typedef enum { FCM_F32 = 0, FCM_BF16 = 1, FCM_I8 = 2 } fcm_dtype;
typedef enum { FCM_NCHW = 0, FCM_NHWC = 1 } fcm_layout;
typedef enum { FCM_ACT_NONE = 0, FCM_ACT_RELU = 1, FCM_ACT_RELU6 = 2 } fcm_act;

/* Module selector for fcm_plan. */
typedef enum {
  FCM_OP_DW_PW = 0,
  FCM_OP_PW_DW = 1,
  FCM_OP_PW_DW_PW = 2,
  FCM_OP_DW = 3,
  FCM_OP_PW = 4,
  FCM_OP_PW_PW = 5
} fcm_op;

/* int8 requantisation of a stage:
 *   q = clamp(rne(acc * mult / 2^shift) + zero_point, qmin, qmax),
 * rne = round half to even, acc = int32 accumulator + int32 bias. int8 activations act on
 * q: RELU and RELU6 clamp it below at zero_point, the code of real 0; RELU6's upper end is
 * qmax, which the caller sets to 6.0 in the output's quantised units (e.g. 24 + zero_point
 * for a scale of 1/4).
 * Asymmetric quantisation: a code q of the stage's output stands for scale * (q -
 * zero_point). The stage that reads it convolves q - zero_point and pads with real 0.
 * The paper states INT8 arithmetic (Sec. III-B) without a quantisation scheme; zero points
 * extend it to asymmetric int8 models and change no module's data movement.
 * Constraints: 0 <= shift <= 62, -128 <= qmin <= qmax <= 127, -128 <= zero_point <= 127.
 * Ignored for float types. */
typedef struct {
  int32_t mult;
  int32_t shift;
  int32_t qmin;
  int32_t qmax;
  int32_t zero_point;
} fcm_requant;

/* One descriptor for every entry point; fields a module does not use are ignored.
 *   fcm_dw_pw:    c_in channels -> DW -> PW -> c_out          (c_mid must equal c_in)
 *   fcm_pw_dw:    c_in -> PW -> c_mid -> DW                   (c_out must equal c_mid)
 *   fcm_pw_dw_pw: c_in -> PW -> c_mid -> DW -> PW -> c_out
 *   fcm_pw_pw:    c_in -> PW -> c_mid -> PW -> c_out on the h x w grid (k, stride, pad ignored)
 *   fcm_dw:       c_in channels, uses act[0], rq[0]
 *   fcm_pw:       c_in -> c_out on the h x w grid (k, stride, pad ignored), act[0], rq[0] */
typedef struct {
  int32_t n, h, w;
  int32_t c_in, c_mid, c_out;
  int32_t k, stride, pad;
  int32_t dtype;   /* fcm_dtype  */
  int32_t layout;  /* fcm_layout */
  int32_t act[3];  /* fcm_act per conv stage, execution order */
  fcm_requant rq[3];
  /* int8 per-channel requantisation of stage i (NULL = per-tensor rq[i]): DEVICE array of
   * 2 x (the stage's output channels) int32, the multipliers then the shifts (shifts in
   * [0, 62]); the clamp range stays rq[i].qmin / qmax. Such descriptors are planned and
   * launched on the first-generation kernels and on the int8 persistent NHWC kernels
   * (DW->PW, DW, PW); an explicit plan on another kernel fails with FCM_EUNSUPPORTED.
   * Ignored for float types. */
  const int32_t* rq_channel[3];
  /* int8 zero point of the input x (the code of real 0, in [-128, 127]); the input of
   * stage i > 0 has the zero point of stage i-1's output, rq[i-1].zero_point. Descriptors
   * with a nonzero zero point anywhere are planned and launched on the first-generation
   * kernels, on the int8 persistent NHWC kernels and on the PW->PW register kernel's
   * instances of at most 192 output channels; an explicit plan on another kernel fails
   * with FCM_EUNSUPPORTED. Ignored for float types. */
  int32_t zp_in;
} fcm_desc;

/* GPU description for the planner (Sec. IV: number of SMs, L1/shared-memory size).
 * On CDNA4 a workgroup's share of the compute unit's LDS plays the role of the paper's
 * L1/shared memory. Pass NULL to fcm_plan for the MI355X defaults
 * (256 CUs, 8 XCDs, wave64, 160 KiB LDS per CU and per workgroup, 4 MiB L2 per XCD,
 * 256 MiB Infinity Cache, 8 TB/s HBM3E). */
typedef struct {
  int32_t num_cus;
  int32_t num_xcds;
  int32_t wave_size;
  int32_t lds_per_wg;   /* bytes */
  int32_t lds_per_cu;   /* bytes */
  int64_t l2_per_xcd;   /* bytes */
  int64_t mall_bytes;   /* bytes */
  double hbm_bytes_per_s;
} fcm_hw_desc;

/* A tiling chosen by fcm_plan (or filled in by the caller and validated at launch).
 * tile_h x tile_w output pixels per workgroup; c_block channels staged per step (the
 * contraction chunk, the depthwise channel block, or for pw_dw_pw / pw_pw the
 * intermediate-channel chunk); co_block channels per workgroup (dw_pw, pw, pw_dw_pw,
 * pw_pw: the last layer's outputs; pw_dw, dw: intermediate / depthwise channels). All
 * byte figures are for the whole call; bytes_paper follows Sec. IV's Eq. 1-4 with the
 * readings listed in the design notes. */
typedef struct {
  int32_t op;            /* fcm_op */
  int32_t tile_h, tile_w;
  int32_t c_block;
  int32_t co_block;
  int32_t variant;       /* compiled kernel family member implementing the plan */
  int32_t waves;         /* waves per workgroup (64 lanes each) */
  int32_t lds_bytes;     /* dynamic LDS per workgroup */
  int32_t workgroups;
  int32_t fuse;          /* planner verdict: 1 if the fused estimate < layer-by-layer */
  int32_t depth;         /* persistent kernels: LDS ring buffers, i.e. items in flight + 1
                            (2..8; 0 on input to fcm_plan_evaluate = the planner's choice) */
  int32_t splits;        /* persistent DW->PW and PW kernels: the channel chunks of each
                            work tile are split over this many workgroups; each writes its
                            partial sums to the caller's workspace and a second kernel
                            adds them in split order, then applies bias, activation and
                            cast. PW->PW register kernel: 1, 2 or 4 waves of a workgroup
                            share a pixel group's intermediate chunks and add their partial
                            sums through LDS in wave order (no workspace).
                            1 = no split; 0 on input to fcm_plan_evaluate = 1 */
  int64_t bytes_ideal;          /* input + weights + output, each once                  */
  int64_t bytes_tiled;          /* per-workgroup loads + stores of this tiling (exact)  */
  int64_t bytes_paper;          /* Eq. 1-4 estimate of this module at this tiling        */
  int64_t bytes_lbl_paper;      /* Eq. 2/3 estimate of the layer-by-layer chain          */
  int64_t bytes_lbl_ideal;      /* layer-by-layer ideal: adds each intermediate twice    */
  double redundancy;     /* recomputed fraction of the first conv (PW->DW halo); 0 else */
} fcm_plan_t;

/* FusePlanner. Chooses the tiling of `op` for `desc` on `hw` (NULL = MI355X) among the
 * tilings the compiled kernels implement. Where a persistent NHWC kernel (or, for PW->PW,
 * the register kernel) implements the shape, the plan with the least time under that
 * kernel's fitted time model wins; otherwise the plan minimises bytes_tiled subject to
 * the LDS limit and to #workgroups >= #CUs where any tiling reaches it (Sec. IV-A
 * constraints), ties broken by more workgroups (up to 2 per CU), then larger tiles.
 * `fuse` is the paper's verdict: the module's Eq. 1-4 estimate against the sum of its
 * layers' (Sec. IV-B). Host-only, deterministic; results are cached per (op, desc, hw).
 * Returns FCM_EINVAL / FCM_EUNSUPPORTED like the launch entry points. */
fcm_status fcm_plan(int32_t op, const fcm_desc* desc, const fcm_hw_desc* hw, fcm_plan_t* out);

/* As fcm_plan, among the plans whose caller workspace (fcm_workspace_bytes) is at most
 * max_workspace_bytes: 0 gives the best plan that needs none, which is what the entry
 * points without a workspace argument launch when their plan is NULL. */
fcm_status fcm_plan_limited(int32_t op, const fcm_desc* desc, const fcm_hw_desc* hw,
                            int64_t max_workspace_bytes, fcm_plan_t* out);

/* The planner's candidate plans for a module, for callers that time them on the device
 * and keep the fastest (Sec. IV runs FusePlanner offline; this hands it the measured
 * choice). Writes at most max_count plans (> 0) to out (HOST array, caller-owned) and
 * their number to *count: out[0] is fcm_plan_limited's choice, then the fastest plan of
 * each other compiled kernel variant under the planner's time models, then the remaining
 * plans, fastest first. Every plan needs at most max_workspace_bytes of caller workspace
 * and can be passed to the module's entry point unchanged. FCM_EINVAL for NULL pointers,
 * max_count <= 0 or a negative limit; the descriptor errors of fcm_plan. */
fcm_status fcm_plan_candidates(int32_t op, const fcm_desc* desc, const fcm_hw_desc* hw,
                               int64_t max_workspace_bytes, fcm_plan_t* out, int32_t max_count,
                               int32_t* count);

/* Evaluate a caller-chosen tiling (plan->op, tile_h, tile_w, c_block, co_block,
 * variant) without searching: fills every other field, or fails with
 * FCM_EUNSUPPORTED if no compiled kernel implements it. */
fcm_status fcm_plan_evaluate(const fcm_desc* desc, const fcm_hw_desc* hw, fcm_plan_t* plan);

/* The planner's estimate of a plan's launch time in seconds (the fitted time model of the
 * plan's kernel family on `hw`, NULL = MI355X), as used by FCM_CHAIN_TIME; 0 on error. */
double fcm_plan_time_estimate(const fcm_desc* desc, const fcm_hw_desc* hw, const fcm_plan_t* plan);

/* DW -> PW module: y = act1(PW(act0(DW(x) + b_dw)) + b_pw).
 *   x [n, c_in, h, w] | w_dw [c_in][k][k] | b_dw [c_in] | w_pw [c_out][c_in] |
 *   b_pw [c_out] | y [n, c_out, h_o, w_o] (layout order as desc->layout).
 * plan may be NULL (the planner's best plan without a workspace, cached); a plan that
 * needs a workspace (splits > 1) fails with FCM_EINVAL: use fcm_dw_pw_ws. */
fcm_status fcm_dw_pw(const fcm_desc* desc, const void* x, const void* w_dw, const void* b_dw,
                     const void* w_pw, const void* b_pw, void* y, const fcm_plan_t* plan,
                     void* stream);

/* DW -> PW module with a caller workspace (Sec. III-A "DWPW"), for plans that split a
 * work tile's channel chunks over several workgroups (fcm_plan_t.splits > 1): their fp32 /
 * int32 partial sums go to `workspace` (DEVICE, 16-byte aligned, caller-owned,
 * workspace_bytes long) and a second kernel adds them in split order before bias,
 * activation and cast, so results equal the unsplit plan's up to the float summation
 * order (int8: bit-exact). plan NULL: the planner's best plan whose workspace fits
 * workspace_bytes (NULL workspace = 0 bytes). An explicit plan needing more than
 * workspace_bytes (fcm_workspace_bytes) fails with FCM_EINVAL. Otherwise as fcm_dw_pw. */
fcm_status fcm_dw_pw_ws(const fcm_desc* desc, const void* x, const void* w_dw, const void* b_dw,
                        const void* w_pw, const void* b_pw, void* y, const fcm_plan_t* plan,
                        void* workspace, int64_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): fcm_dw_pw_ws with the workspace taken
 * from a fixed device array of FCM_NOALLOC_SCRATCH_BYTES that the library holds on each
 * GPU it runs on (from module load until the process ends) instead of from the caller.
 * It allocates nothing and calls no allocating routine. plan NULL: the planner's best
 * plan whose workspace fits the array; an explicit plan needing more fails with
 * FCM_EINVAL. Every call on one GPU shares that GPU's array, so calls that overlap on one
 * GPU (e.g. on two streams) race; the array keeps the last call's partial sums and needs
 * no clearing (each split plan writes all it reads). FCM_EDEVICE if the runtime cannot
 * resolve the array's device address. Otherwise as fcm_dw_pw. */
#define FCM_NOALLOC_SCRATCH_BYTES (16u << 20)
fcm_status fcm_dw_pw_noalloc(const fcm_desc* desc, const void* x, const void* w_dw, const void* b_dw,
                             const void* w_pw, const void* b_pw, void* y, const fcm_plan_t* plan,
                             void* stream);

/* Device workspace bytes `plan` needs (its partial sums when it splits channel chunks over
 * workgroups; 0 for every other plan), or -1 for an invalid descriptor or plan. */
int64_t fcm_workspace_bytes(const fcm_desc* desc, const fcm_plan_t* plan);

/* PW -> DW module: y = act1(DW(pad0(act0(PW(x) + b_pw))) + b_dw); the DW input is zero
 * outside the image (never act0(b_pw)).
 *   x [n, c_in, h, w] | w_pw [c_mid][c_in] | b_pw [c_mid] | w_dw [c_mid][k][k] |
 *   b_dw [c_mid] | y [n, c_mid, h_o, w_o]. */
fcm_status fcm_pw_dw(const fcm_desc* desc, const void* x, const void* w_pw, const void* b_pw,
                     const void* w_dw, const void* b_dw, void* y, const fcm_plan_t* plan,
                     void* stream);

/* PW -> DW -> PW module (inverted residual, no skip connection):
 *   x [n, c_in, h, w] | w_pw1 [c_mid][c_in] | w_dw [c_mid][k][k] | w_pw2 [c_out][c_mid] |
 *   biases [c_mid], [c_mid], [c_out] | y [n, c_out, h_o, w_o]. */
fcm_status fcm_pw_dw_pw(const fcm_desc* desc, const void* x, const void* w_pw1,
                        const void* b_pw1, const void* w_dw, const void* b_dw,
                        const void* w_pw2, const void* b_pw2, void* y, const fcm_plan_t* plan,
                        void* stream);

/* PW -> PW (the paper's PwPw module, Sec. III-A): y = cast(act1(P2 * cast(act0(P1 * x + b1))
 * + b2)), P1 [c_mid][c_in], P2 [c_out][c_mid]; the spatial size is unchanged (k, stride and
 * pad are ignored). desc->act[0]/rq[0] belong to the first layer, act[1]/rq[1] to the
 * second. Same conventions and errors as fcm_dw_pw. */
fcm_status fcm_pw_pw(const fcm_desc* desc, const void* x, const void* w_pw1, const void* b_pw1,
                     const void* w_pw2, const void* b_pw2, void* y, const fcm_plan_t* plan, void* stream);

/* Single depthwise layer (layer-by-layer baseline): y [n, c_in, h_o, w_o]. */
fcm_status fcm_dw(const fcm_desc* desc, const void* x, const void* w_dw, const void* b_dw,
                  void* y, const fcm_plan_t* plan, void* stream);

/* Single pointwise layer (layer-by-layer baseline): y [n, c_out, h, w]. */
fcm_status fcm_pw(const fcm_desc* desc, const void* x, const void* w_pw, const void* b_pw,
                  void* y, const fcm_plan_t* plan, void* stream);

/* Single pointwise layer with a caller workspace for split plans (as fcm_dw_pw_ws). */
fcm_status fcm_pw_ws(const fcm_desc* desc, const void* x, const void* w_pw, const void* b_pw,
                     void* y, const fcm_plan_t* plan, void* workspace, int64_t workspace_bytes,
                     void* stream);

/* ------------------------------------------------------------------------------------
 * Chains of layers: FusePlanner over a network (Sec. IV: FCMs and layer-by-layer kernels
 * "used to derive complete CNN execution plans"; Sec. V reports the share of conv layers
 * fused in whole models).
 *
 * A chain is a sequence of DW and PW layers, each consuming the previous layer's output
 * (no skip connections). fcm_chain_plan partitions it into groups, each run as one
 * kernel: a single layer (fcm_dw / fcm_pw) or a fused module over adjacent layers
 * (DW->PW, PW->DW, PW->PW, PW->DW->PW). Every candidate group is planned with fcm_plan;
 * dynamic programming over the chain picks the partition of least total cost. With
 * FCM_CHAIN_BYTES the cost is the paper's global-memory-access estimate (bytes_paper,
 * Eq. 1-4), so a pair is fused exactly when the module's estimate is below the sum of
 * its layers' (Sec. IV-B), applied to the whole chain at once; ties keep layers apart.
 * FCM_CHAIN_TIME uses the fitted time models of the kernels the plans launch (plans of
 * kernels without one: their bytes at the HBM rate plus a launch). FCM_CHAIN_UNFUSED
 * runs every layer alone (the layer-by-layer baseline).
 * ------------------------------------------------------------------------------------ */

#define FCM_CHAIN_MAX_LAYERS 128

typedef enum { FCM_LAYER_DW = 0, FCM_LAYER_PW = 1 } fcm_layer_kind;
typedef enum { FCM_CHAIN_BYTES = 0, FCM_CHAIN_TIME = 1, FCM_CHAIN_UNFUSED = 2 } fcm_chain_objective;

/* One layer: conv -> +bias -> act -> cast (int8: requantised by rq). */
typedef struct {
  int32_t kind;            /* fcm_layer_kind */
  int32_t c_out;           /* PW: output channels; DW: ignored (equals its input channels) */
  int32_t k, stride, pad;  /* DW geometry (as fcm_desc); ignored for PW */
  int32_t act;             /* fcm_act */
  fcm_requant rq;          /* FCM_I8 only */
} fcm_layer;

typedef struct {
  int32_t n, h, w, c;      /* input of the first layer */
  int32_t dtype;           /* fcm_dtype, the whole chain */
  int32_t layout;          /* fcm_layout, the whole chain */
  int32_t zp_in;           /* FCM_I8: zero point of the chain input (layer i > 0 reads
                              layer i-1's output zero point, layers[i-1].rq.zero_point) */
  int32_t num_layers;      /* 1 .. FCM_CHAIN_MAX_LAYERS */
  fcm_layer layers[FCM_CHAIN_MAX_LAYERS];
} fcm_chain_desc;

typedef struct {
  int32_t objective;                      /* fcm_chain_objective it was made for */
  int32_t num_groups;
  int32_t first[FCM_CHAIN_MAX_LAYERS];    /* first layer of group g */
  int32_t op[FCM_CHAIN_MAX_LAYERS];       /* fcm_op of group g (its layers: first[g] ..) */
  fcm_plan_t plan[FCM_CHAIN_MAX_LAYERS];  /* plan of group g */
  int32_t fused_layers;                   /* layers that run inside fused modules */
  int64_t act_bytes_max;                  /* largest activation passed between groups */
  int64_t bytes_paper, bytes_lbl_paper;   /* Eq. 1-4 totals: this partition, every layer alone */
  double time_est, time_lbl_est;          /* time-model totals (seconds), same two */
} fcm_chain_plan_t;

/* Plan a chain (hw: NULL = MI355X). Fails with FCM_EINVAL for an invalid chain (sizes,
 * geometry, requantisation, as the single-layer entry points) and FCM_EUNSUPPORTED if
 * some layer has no compiled kernel at all. Host-only, deterministic. */
fcm_status fcm_chain_plan(const fcm_chain_desc* chain, int32_t objective, const fcm_hw_desc* hw,
                          fcm_chain_plan_t* out);

/* Device bytes fcm_chain_run needs in `workspace` for `plan` (two activation buffers,
 * each aligned to 256 bytes; 0 when the chain is one group). */
int64_t fcm_chain_workspace_bytes(const fcm_chain_plan_t* plan);

/* Run a planned chain on `stream`: x is the chain input, y the last layer's output
 * (shapes from the chain and each layer's geometry, layout chain->layout); weights[i],
 * biases[i] belong to layer i (canonical layouts as the single-layer entry points;
 * biases[i] may be NULL). `workspace` (device, fcm_chain_workspace_bytes(plan) bytes,
 * caller-owned, may be NULL when that is 0) holds the activations between groups. Chain
 * plans use no split plans, so that is all the device memory a chain needs.
 * Errors are those of the group launches; a failing group stops the chain. */
fcm_status fcm_chain_run(const fcm_chain_desc* chain, const fcm_chain_plan_t* plan, const void* x,
                         const void* const* weights, const void* const* biases, void* workspace, void* y,
                         void* stream);

/* Fold an inference-mode batch normalisation that follows a convolution into that
 * convolution's weights and bias (an FCM stage is convolution -> normalisation ->
 * activation, Sec. III-A; the kernels take the normalisation folded). For output channel o:
 *   s_o = gamma[o] / sqrt(var[o] + eps),  w_out[o][j] = w[o][j] * s_o,
 *   b_out[o] = (b[o] - mean[o]) * s_o + beta[o]            (b may be NULL: zero)
 * computed in double, rounded to float. w holds c_out rows of `row` floats (depthwise
 * [c][k][k]: row = k*k; pointwise [c_out][c_in]: row = c_in). HOST pointers; w_out / b_out
 * may alias w / b. Float models only (int8 folds into its requantisation instead).
 * FCM_EINVAL for NULL arrays, non-positive sizes, eps < 0 or var + eps <= 0. */
fcm_status fcm_fold_batchnorm(int32_t c_out, int32_t row, const float* w, const float* b, const float* gamma,
                              const float* beta, const float* mean, const float* var, float eps, float* w_out,
                              float* b_out);

/* Human-readable name of a status code (static storage). */
const char* fcm_status_string(fcm_status status);

/* Detail of the last failure on the calling thread ("" if none). */
const char* fcm_last_error(void);

/* Library version string. */
const char* fcm_version(void);

/* Name of a compiled kernel variant (as fcm_plan_t.variant), e.g. for matching profiler
 * output to plans; NULL if out of range. Static storage. */
const char* fcm_variant_name(int32_t variant);

/* Number of compiled kernel variants. */
int32_t fcm_variant_count(void);

#ifdef __cplusplus
}
#endif

#endif /* FCM_H_ */
