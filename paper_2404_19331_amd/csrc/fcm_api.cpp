// fcm_api.cpp -- the C ABI of libfcm.so: argument validation, plan lookup, kernel
// argument marshalling and launch.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "fcm_host.h"

namespace fcm {

static thread_local std::string g_last_error;

fcm_status fail(fcm_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

void int8_features(int op, const fcm_desc* d, int* zp, int* pc) {
  *zp = *pc = 0;
  if (!d || d->dtype != FCM_I8) return;
  const int stages = op == FCM_OP_PW_DW_PW ? 3 : ((op == FCM_OP_DW || op == FCM_OP_PW) ? 1 : 2);
  *zp = d->zp_in != 0;
  for (int i = 0; i < stages; ++i) {
    if (d->rq_channel[i]) *pc = 1;
    if (d->rq[i].zero_point != 0) *zp = 1;
  }
}

// int8 features not every kernel implements: per-channel requantisation (first-generation
// and int8 persistent kernels) and zero points (those and the PW->PW register kernel).
int kernel_set(int op, const fcm_desc* d) {
  int zp, pc;
  int8_features(op, d, &zp, &pc);
  return pc ? KSET_PC : (zp ? KSET_REG : KSET_ALL);
}

static const char* kset_message(int kset) {
  return kset == KSET_PC ? "per-channel requantisation runs on the first-generation and int8 persistent kernels only"
                         : "zero points run on the first-generation, int8 persistent and PW->PW register kernels only";
}

const Variant* all_variants(int* count) {
  static std::vector<Variant> all = [] {
    std::vector<Variant> v;
    const Variant* (*fns[])(int*) = {variants_dwpw_f32, variants_dwpw_bf16, variants_dwpw_i8, variants_pwdw,
                                     variants_pwdwpw,
                                     variants_v3_dwpw_bf16_s1, variants_v3_dwpw_bf16_s2, variants_v3_dwpw_f32,
                                     variants_v3_dwpw_i8, variants_v3_pw, variants_v3_pw_f32, variants_v3_pw_i8,
                                     variants_v3_dw_bf16, variants_v3_dw_f32, variants_v3_dw_i8,
                                     variants_v4_pwpw_i8, variants_v4_pwpw_bf16, variants_v4_pwpw_f32,
                                     variants_v5_dwpw_bf16_s1, variants_v5_dwpw_bf16_s2, variants_v5_pwdw_bf16,
                                     variants_v6_f32, variants_v7_bf16};
    for (auto fn : fns) {
      int n = 0;
      const Variant* t = fn(&n);
      v.insert(v.end(), t, t + n);
    }
    return v;
  }();
  *count = (int)all.size();
  return all.data();
}

static bool uses_dw(int op) { return op != FCM_OP_PW && op != FCM_OP_PW_PW; }

fcm_status validate(int op, const fcm_desc* d) {
  if (op < FCM_OP_DW_PW || op > FCM_OP_PW_PW) return fail(FCM_EINVAL, "unknown module");
  if (!d) return fail(FCM_EINVAL, "descriptor is NULL");
  if (d->n <= 0 || d->h <= 0 || d->w <= 0 || d->c_in <= 0)
    return fail(FCM_EINVAL, "n, h, w and c_in must be positive");
  if (d->dtype < FCM_F32 || d->dtype > FCM_I8) return fail(FCM_EINVAL, "unknown dtype");
  if (d->layout != FCM_NCHW && d->layout != FCM_NHWC) return fail(FCM_EINVAL, "unknown layout");
  const int stages = op == FCM_OP_PW_DW_PW ? 3 : ((op == FCM_OP_DW || op == FCM_OP_PW) ? 1 : 2);
  for (int i = 0; i < stages; ++i) {
    if (d->act[i] < FCM_ACT_NONE || d->act[i] > FCM_ACT_RELU6) return fail(FCM_EINVAL, "unknown activation");
    if (d->dtype == FCM_I8) {
      const fcm_requant& r = d->rq[i];
      if (r.shift < 0 || r.shift > 62) return fail(FCM_EINVAL, "requant shift must be in [0, 62]");
      if (r.qmin < -128 || r.qmax > 127 || r.qmin > r.qmax)
        return fail(FCM_EINVAL, "requant range must satisfy -128 <= qmin <= qmax <= 127");
      if (r.zero_point < -128 || r.zero_point > 127) return fail(FCM_EINVAL, "zero points must be in [-128, 127]");
    }
  }
  if (d->dtype == FCM_I8 && (d->zp_in < -128 || d->zp_in > 127))
    return fail(FCM_EINVAL, "zero points must be in [-128, 127]");
  switch (op) {
    case FCM_OP_DW_PW:
      if (d->c_out <= 0) return fail(FCM_EINVAL, "c_out must be positive");
      if (d->c_mid != d->c_in) return fail(FCM_EINVAL, "dw_pw: c_mid must equal c_in");
      break;
    case FCM_OP_PW_DW:
      if (d->c_mid <= 0) return fail(FCM_EINVAL, "c_mid must be positive");
      if (d->c_out != d->c_mid) return fail(FCM_EINVAL, "pw_dw: c_out must equal c_mid");
      break;
    case FCM_OP_PW_DW_PW:
    case FCM_OP_PW_PW:
      if (d->c_mid <= 0 || d->c_out <= 0) return fail(FCM_EINVAL, "c_mid and c_out must be positive");
      break;
    case FCM_OP_PW:
      if (d->c_out <= 0) return fail(FCM_EINVAL, "c_out must be positive");
      break;
    default:
      break;
  }
  if (uses_dw(op)) {
    if (d->k <= 0 || d->stride <= 0 || d->pad < 0) return fail(FCM_EINVAL, "k and stride must be positive, pad >= 0");
    if (d->pad >= d->k) return fail(FCM_EINVAL, "pad must be smaller than k");
    if (d->h + 2 * d->pad < d->k || d->w + 2 * d->pad < d->k) return fail(FCM_EINVAL, "output would be empty");
    if (d->k != 3 && d->k != 5) return fail(FCM_EUNSUPPORTED, "depthwise k must be 3 or 5");
    if (d->stride != 1 && d->stride != 2) return fail(FCM_EUNSUPPORTED, "depthwise stride must be 1 or 2");
  }
  const int64_t big = (int64_t)d->n * d->h * d->w;
  const int64_t cmax = std::max(std::max(d->c_in, d->c_mid), d->c_out);
  if (big * cmax > (int64_t)1 << 40) return fail(FCM_EUNSUPPORTED, "tensor too large");
  return FCM_OK;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }


// Compute units of the current device (queried once per device).
static int device_cus() {
  static std::mutex mu;
  static std::vector<int> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return default_hw().num_cus;
  std::lock_guard<std::mutex> lock(mu);
  if ((int)cache.size() <= dev) cache.resize(dev + 1, 0);
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = default_hw().num_cus;
    cache[dev] = n;
  }
  return cache[dev];
}

static fcm_status check_alignment(const void* p, int elt, const char* what) {
  if (p && ((uintptr_t)p % (uintptr_t)elt) != 0)
    return fail(FCM_EINVAL, std::string(what) + " is not aligned to its element size");
  return FCM_OK;
}

struct Tensors {
  const void* x;
  const void* w[3];
  const void* b[3];
  void* y;
};

// ws / ws_bytes: the caller's device workspace (split plans keep their partial sums
// there); NULL / 0 = none, and then only plans that need none are used or accepted.
static fcm_status run(int op, const fcm_desc* d, const Tensors& t, const fcm_plan_t* plan_in, void* ws,
                      int64_t ws_bytes, void* stream) {
  if (ws_bytes < 0) return fail(FCM_EINVAL, "workspace size must not be negative");
  if (ws && ((uintptr_t)ws & 15u)) return fail(FCM_EINVAL, "workspace must be 16-byte aligned");
  if (!ws) ws_bytes = 0;
  fcm_status st = validate(op, d);
  if (st != FCM_OK) return st;
  const int nw = op == FCM_OP_PW_DW_PW ? 3 : ((op == FCM_OP_DW || op == FCM_OP_PW) ? 1 : 2);
  if (!t.x || !t.y) return fail(FCM_EINVAL, "x and y must not be NULL");
  for (int i = 0; i < nw; ++i)
    if (!t.w[i]) return fail(FCM_EINVAL, "weights must not be NULL");
  const Geom g = geometry(op, d);
  const int e = g.elt;
  if ((st = check_alignment(t.x, e, "x")) || (st = check_alignment(t.y, e, "y"))) return st;
  for (int i = 0; i < nw; ++i) {
    if ((st = check_alignment(t.w[i], e, "weights"))) return st;
    if ((st = check_alignment(t.b[i], 4, "bias"))) return st;
  }

  const fcm_hw_desc hw = default_hw();
  // LDS-DMA kernels need 16-byte aligned tensors
  bool aligned = aligned16(t.x) && aligned16(t.y);
  for (int i = 0; i < nw; ++i) aligned = aligned && aligned16(t.w[i]);
  // the kernels the descriptor's int8 features allow, and of those the ones the tensors'
  // alignment allows
  const int feat = kernel_set(op, d);
  const int kset = aligned ? feat : KSET_FIRST;
  fcm_plan_t p;
  if (plan_in) {
    if (plan_in->op != op) return fail(FCM_EINVAL, "plan was made for another module");
    p = *plan_in;
    if ((st = evaluate_plan(g, d, hw, &p)) != FCM_OK) return st;
    if (!variant_in_set(p.variant, kset))
      return fail(FCM_EUNSUPPORTED, !variant_in_set(p.variant, feat) ? kset_message(feat)
                                                                       : "plan's kernel needs 16-byte aligned tensors");
  } else {
    if ((st = find_plan(op, d, &hw, &p, kset, ws_bytes)) != FCM_OK) return st;
  }
  const int64_t need = plan_workspace_bytes(g, p);
  if (need > ws_bytes)
    return fail(FCM_EINVAL, "the plan splits its channel chunks and needs " + std::to_string(need) +
                                " bytes of caller workspace (fcm_workspace_bytes; pass it to the _ws entry point)");
  int nv = 0;
  const Variant* vs = all_variants(&nv);
  const Variant& v = vs[p.variant];

  KArgs a;
  memset(&a, 0, sizeof(a));
  a.x = t.x;
  a.y = t.y;
  a.w1 = t.w[0];
  a.b1 = t.b[0];
  a.w2 = t.w[1];
  a.b2 = t.b[1];
  a.w3 = t.w[2];
  a.b3 = t.b[2];
  a.N = g.n;
  a.H = g.h;
  a.W = g.w;
  a.Ci = g.ci;
  a.Cm = g.cm;
  a.Co = g.co;
  a.Ho = g.ho;
  a.Wo = g.wo;
  a.pad = g.pad;
  a.layout = d->layout;
  a.TH = p.tile_h;
  a.TW = p.tile_w;
  a.CB = p.c_block;
  a.COB = p.co_block;
  a.tiles_y = ceil_div(g.ho, p.tile_h);
  a.tiles_x = ceil_div(g.wo, p.tile_w);
  const int last = (g.family == FAM_PWDW || g.family == FAM_DW) ? g.cm : g.co;
  a.n_cb = ceil_div(last, p.co_block);
  const bool i8 = d->dtype == FCM_I8;
  for (int i = 0; i < 3; ++i) {
    a.rqc[i] = (i8 && i < nw) ? d->rq_channel[i] : nullptr;
    a.act[i] = d->act[i];
    a.rq[i].mult = d->rq[i].mult;
    a.rq[i].shift = d->rq[i].shift;
    a.rq[i].qmin = d->rq[i].qmin;
    a.rq[i].qmax = d->rq[i].qmax;
    a.rq[i].zp = i8 ? d->rq[i].zero_point : 0;
    a.zin[i] = !i8 ? 0 : (i == 0 ? d->zp_in : d->rq[i - 1].zero_point);
  }
  // vector paths: 16-byte aligned base and 16-byte multiple rows
  const int xc = g.family == FAM_DW ? g.cm : g.ci;
  a.vec_x = aligned16(t.x) && (xc * e) % 16 == 0;
  a.vec_y = aligned16(t.y) && (last * e) % 16 == 0;
  switch (g.family) {
    case FAM_DWPW: a.vec_w2 = aligned16(t.w[1]) && (g.ci * e) % 16 == 0; break;
    case FAM_PW: a.vec_w1 = aligned16(t.w[0]) && (g.ci * e) % 16 == 0; break;
    case FAM_PWDW: a.vec_w1 = aligned16(t.w[0]) && (g.ci * e) % 16 == 0; break;
    case FAM_PWDWPW:
      a.vec_w1 = aligned16(t.w[0]) && (g.ci * e) % 16 == 0;
      a.vec_w3 = aligned16(t.w[2]) && (g.cm * e) % 16 == 0;
      break;
    case FAM_PWPW:  // second PW weights in w2, its vector flag in vec_w3
      a.vec_w1 = aligned16(t.w[0]) && (g.ci * e) % 16 == 0;
      a.vec_w3 = aligned16(t.w[1]) && (g.cm * e) % 16 == 0;
      break;
    default: break;
  }
  a.nwork = a.N * a.tiles_y * a.tiles_x * a.n_cb;
  a.splits = 1;
  if (v.gen == 3 && p.splits > 1) {
    a.ws = ws;
    a.splits = p.splits;
    a.nwork *= p.splits;  // work units
  }
  if (v.gen == 4) {
    // PW -> PW register kernel: pixel groups, each on `splits` waves of one workgroup
    a.nwork = (int)ceil_div((int64_t)g.n * g.h * g.w, (int64_t)v.max_p);
    a.splits = p.splits;
    a.vec_w2 = aligned16(t.w[1]) && (g.cm * e) % 16 == 0;
  }
  a.cus = device_cus();
  a.grid_cap = (v.gen == 3 || v.gen == 5 || v.gen == 7) ? p.workgroups : 0;
  a.depth = p.depth;
  if (v.gen >= 2) {
    a.L = LdsLayout{};
    a.L.bytes = p.lds_bytes;
  } else switch (g.family) {
    case FAM_DWPW:
    case FAM_PW:
      a.L = lds_layout_dwpw(g.dtype, g.k, g.s, g.family == FAM_DWPW, p.tile_h, p.tile_w, p.c_block, p.co_block);
      break;
    case FAM_PWDW:
    case FAM_DW:
      a.L = lds_layout_pwdw(g.dtype, g.k, g.s, g.family == FAM_PWDW, p.tile_h, p.tile_w, p.c_block, p.co_block);
      break;
    default:
      a.L = lds_layout_pwdwpw(g.dtype, g.k, g.s, p.tile_h, p.tile_w, g.ci, p.c_block, p.co_block);
      break;
  }
  const int rc = v.launch(a, p.workgroups, stream);
  if (rc != 0)
    return fail(FCM_EDEVICE, std::string("kernel launch failed: ") + hipGetErrorString((hipError_t)rc) + " (" +
                                 v.name + ")");
  return FCM_OK;
}

fcm_status launch_module(int op, const fcm_desc* d, const void* x, const void* const* w, const void* const* b,
                         void* y, const fcm_plan_t* plan, void* ws, int64_t ws_bytes, void* stream) {
  Tensors t = {x, {w[0], w[1], w[2]}, {b[0], b[1], b[2]}, y};
  return run(op, d, t, plan, ws, ws_bytes, stream);
}

}  // namespace fcm

using namespace fcm;

extern "C" {

fcm_status fcm_plan(int32_t op, const fcm_desc* desc, const fcm_hw_desc* hw, fcm_plan_t* out) {
  if (!out) return fail(FCM_EINVAL, "output plan is NULL");
  fcm_status st = validate(op, desc);
  if (st != FCM_OK) return st;
  return find_plan(op, desc, hw, out, kernel_set(op, desc));
}

fcm_status fcm_plan_limited(int32_t op, const fcm_desc* desc, const fcm_hw_desc* hw, int64_t max_workspace_bytes,
                            fcm_plan_t* out) {
  if (!out) return fail(FCM_EINVAL, "output plan is NULL");
  if (max_workspace_bytes < 0) return fail(FCM_EINVAL, "workspace limit must not be negative");
  fcm_status st = validate(op, desc);
  if (st != FCM_OK) return st;
  return find_plan(op, desc, hw, out, kernel_set(op, desc), max_workspace_bytes);
}

fcm_status fcm_plan_candidates(int32_t op, const fcm_desc* desc, const fcm_hw_desc* hw, int64_t max_workspace_bytes,
                               fcm_plan_t* out, int32_t max_count, int32_t* count) {
  if (!out || !count) return fail(FCM_EINVAL, "output plans or count is NULL");
  *count = 0;
  if (max_count <= 0) return fail(FCM_EINVAL, "max_count must be positive");
  if (max_workspace_bytes < 0) return fail(FCM_EINVAL, "workspace limit must not be negative");
  fcm_status st = validate(op, desc);
  if (st != FCM_OK) return st;
  int n = 0;
  st = find_candidates(op, desc, hw, kernel_set(op, desc), max_workspace_bytes, out, max_count, &n);
  *count = n;
  return st;
}

fcm_status fcm_plan_evaluate(const fcm_desc* desc, const fcm_hw_desc* hw, fcm_plan_t* plan) {
  if (!plan) return fail(FCM_EINVAL, "plan is NULL");
  fcm_status st = validate(plan->op, desc);
  if (st != FCM_OK) return st;
  const fcm_hw_desc h = hw ? *hw : default_hw();
  const Geom g = geometry(plan->op, desc);
  st = evaluate_plan(g, desc, h, plan);
  if (st != FCM_OK) return st;
  const int kset = kernel_set(plan->op, desc);
  if (!variant_in_set(plan->variant, kset)) return fail(FCM_EUNSUPPORTED, kset_message(kset));
  // the layer-by-layer figures and the verdict come from the searched plan
  fcm_plan_t ref;
  st = find_plan(plan->op, desc, &h, &ref, kset);
  if (st != FCM_OK) return st;
  plan->bytes_lbl_paper = ref.bytes_lbl_paper;
  plan->bytes_lbl_ideal = ref.bytes_lbl_ideal;
  plan->fuse = plan->bytes_paper < plan->bytes_lbl_paper ? 1 : 0;
  if (plan->op == FCM_OP_DW || plan->op == FCM_OP_PW) plan->fuse = 0;
  return FCM_OK;
}

double fcm_plan_time_estimate(const fcm_desc* desc, const fcm_hw_desc* hw, const fcm_plan_t* plan) {
  if (!plan || validate(plan->op, desc) != FCM_OK) return 0.0;
  const fcm_hw_desc H = hw ? *hw : default_hw();
  return plan_time_estimate(geometry(plan->op, desc), *plan, H);
}

fcm_status fcm_fold_batchnorm(int32_t c_out, int32_t row, const float* w, const float* b, const float* gamma,
                              const float* beta, const float* mean, const float* var, float eps, float* w_out,
                              float* b_out) {
  if (c_out <= 0 || row <= 0) return fail(FCM_EINVAL, "fold_batchnorm: c_out and row must be positive");
  if (!w || !gamma || !beta || !mean || !var || !w_out || !b_out)
    return fail(FCM_EINVAL, "fold_batchnorm: NULL array");
  if (!(eps >= 0.0f)) return fail(FCM_EINVAL, "fold_batchnorm: eps must be >= 0");
  for (int32_t o = 0; o < c_out; ++o)
    if (!((double)var[o] + (double)eps > 0.0)) return fail(FCM_EINVAL, "fold_batchnorm: var + eps must be > 0");
  for (int32_t o = 0; o < c_out; ++o) {
    const double sc = (double)gamma[o] / std::sqrt((double)var[o] + (double)eps);
    const double bo = b ? (double)b[o] : 0.0;
    for (int32_t j = 0; j < row; ++j) {
      const size_t i = (size_t)o * row + j;
      w_out[i] = (float)((double)w[i] * sc);
    }
    b_out[o] = (float)((bo - (double)mean[o]) * sc + (double)beta[o]);
  }
  return FCM_OK;
}

fcm_status fcm_dw_pw(const fcm_desc* desc, const void* x, const void* w_dw, const void* b_dw, const void* w_pw,
                     const void* b_pw, void* y, const fcm_plan_t* plan, void* stream) {
  Tensors t = {x, {w_dw, w_pw, nullptr}, {b_dw, b_pw, nullptr}, y};
  return run(FCM_OP_DW_PW, desc, t, plan, nullptr, 0, stream);
}

fcm_status fcm_dw_pw_ws(const fcm_desc* desc, const void* x, const void* w_dw, const void* b_dw, const void* w_pw,
                        const void* b_pw, void* y, const fcm_plan_t* plan, void* workspace, int64_t workspace_bytes,
                        void* stream) {
  Tensors t = {x, {w_dw, w_pw, nullptr}, {b_dw, b_pw, nullptr}, y};
  return run(FCM_OP_DW_PW, desc, t, plan, workspace, workspace_bytes, stream);
}

fcm_status fcm_pw_dw(const fcm_desc* desc, const void* x, const void* w_pw, const void* b_pw, const void* w_dw,
                     const void* b_dw, void* y, const fcm_plan_t* plan, void* stream) {
  Tensors t = {x, {w_pw, w_dw, nullptr}, {b_pw, b_dw, nullptr}, y};
  return run(FCM_OP_PW_DW, desc, t, plan, nullptr, 0, stream);
}

fcm_status fcm_pw_dw_pw(const fcm_desc* desc, const void* x, const void* w_pw1, const void* b_pw1, const void* w_dw,
                        const void* b_dw, const void* w_pw2, const void* b_pw2, void* y, const fcm_plan_t* plan,
                        void* stream) {
  Tensors t = {x, {w_pw1, w_dw, w_pw2}, {b_pw1, b_dw, b_pw2}, y};
  return run(FCM_OP_PW_DW_PW, desc, t, plan, nullptr, 0, stream);
}

fcm_status fcm_dw(const fcm_desc* desc, const void* x, const void* w_dw, const void* b_dw, void* y,
                  const fcm_plan_t* plan, void* stream) {
  Tensors t = {x, {w_dw, nullptr, nullptr}, {b_dw, nullptr, nullptr}, y};
  return run(FCM_OP_DW, desc, t, plan, nullptr, 0, stream);
}

fcm_status fcm_pw_pw(const fcm_desc* desc, const void* x, const void* w_pw1, const void* b_pw1, const void* w_pw2,
                     const void* b_pw2, void* y, const fcm_plan_t* plan, void* stream) {
  Tensors t = {x, {w_pw1, w_pw2, nullptr}, {b_pw1, b_pw2, nullptr}, y};
  return run(FCM_OP_PW_PW, desc, t, plan, nullptr, 0, stream);
}

fcm_status fcm_chain_run(const fcm_chain_desc* chain, const fcm_chain_plan_t* plan, const void* x,
                         const void* const* weights, const void* const* biases, void* workspace, void* y,
                         void* stream) {
  if (!plan) return fail(FCM_EINVAL, "chain plan is NULL");
  if (!weights) return fail(FCM_EINVAL, "weights array is NULL");
  std::vector<int> h(FCM_CHAIN_MAX_LAYERS + 1), w(FCM_CHAIN_MAX_LAYERS + 1), ch(FCM_CHAIN_MAX_LAYERS + 1);
  fcm_status st = chain_shapes(chain, h.data(), w.data(), ch.data());
  if (st != FCM_OK) return st;
  // the plan must cover the chain exactly, group after group
  if (plan->num_groups < 1 || plan->num_groups > chain->num_layers) return fail(FCM_EINVAL, "chain plan: bad group count");
  std::vector<fcm_desc> descs(plan->num_groups);
  int next = 0;
  for (int g = 0; g < plan->num_groups; ++g) {
    if (plan->first[g] != next || next >= chain->num_layers ||
        chain_group_desc(chain, h.data(), w.data(), ch.data(), next, plan->op[g], &descs[g]) != FCM_OK)
      return fail(FCM_EINVAL, "chain plan does not match the chain");
    next += op_layers(plan->op[g]);
  }
  if (next != chain->num_layers) return fail(FCM_EINVAL, "chain plan does not match the chain");
  const int64_t half = fcm_chain_workspace_bytes(plan) / 2;
  if (plan->num_groups > 1 && !workspace) return fail(FCM_EINVAL, "chain needs a workspace");
  const void* in = x;
  for (int g = 0; g < plan->num_groups; ++g) {
    const int first = plan->first[g], op = plan->op[g], nl = op_layers(op);
    const fcm_desc& d = descs[g];
    const int64_t e = chain->dtype == FCM_F32 ? 4 : (chain->dtype == FCM_BF16 ? 2 : 1);
    if ((int64_t)chain->n * h[first + nl] * w[first + nl] * ch[first + nl] * e > half && g + 1 < plan->num_groups)
      return fail(FCM_EINVAL, "chain plan's workspace size does not fit the chain");
    void* out = g + 1 == plan->num_groups ? y : (char*)workspace + (g % 2) * half;
    Tensors t = {in, {nullptr, nullptr, nullptr}, {nullptr, nullptr, nullptr}, out};
    for (int i = 0; i < nl; ++i) {
      t.w[i] = weights[first + i];
      t.b[i] = biases ? biases[first + i] : nullptr;
    }
    if ((st = run(op, &d, t, &plan->plan[g], nullptr, 0, stream)) != FCM_OK) return st;
    in = out;
  }
  return FCM_OK;
}

fcm_status fcm_pw(const fcm_desc* desc, const void* x, const void* w_pw, const void* b_pw, void* y,
                  const fcm_plan_t* plan, void* stream) {
  Tensors t = {x, {w_pw, nullptr, nullptr}, {b_pw, nullptr, nullptr}, y};
  return run(FCM_OP_PW, desc, t, plan, nullptr, 0, stream);
}

fcm_status fcm_pw_ws(const fcm_desc* desc, const void* x, const void* w_pw, const void* b_pw, void* y,
                     const fcm_plan_t* plan, void* workspace, int64_t workspace_bytes, void* stream) {
  Tensors t = {x, {w_pw, nullptr, nullptr}, {b_pw, nullptr, nullptr}, y};
  return run(FCM_OP_PW, desc, t, plan, workspace, workspace_bytes, stream);
}

int64_t fcm_workspace_bytes(const fcm_desc* desc, const fcm_plan_t* plan) {
  if (!plan) {
    fail(FCM_EINVAL, "plan is NULL");
    return -1;
  }
  if (validate(plan->op, desc) != FCM_OK) return -1;
  const Geom g = geometry(plan->op, desc);
  fcm_plan_t p = *plan;
  if (evaluate_plan(g, desc, default_hw(), &p) != FCM_OK) return -1;
  return plan_workspace_bytes(g, p);
}

const char* fcm_status_string(fcm_status status) {
  switch (status) {
    case FCM_OK: return "FCM_OK";
    case FCM_EINVAL: return "FCM_EINVAL: invalid argument";
    case FCM_EUNSUPPORTED: return "FCM_EUNSUPPORTED: not supported by the compiled kernels";
    case FCM_EDEVICE: return "FCM_EDEVICE: HIP error";
  }
  return "unknown fcm_status";
}

const char* fcm_last_error(void) { return g_last_error.c_str(); }

const char* fcm_version(void) { return "fcm 0.1.0 (gfx950)"; }

const char* fcm_variant_name(int32_t variant) {
  int nv = 0;
  const Variant* vs = all_variants(&nv);
  return (variant >= 0 && variant < nv) ? vs[variant].name : nullptr;
}

int32_t fcm_variant_count(void) {
  int nv = 0;
  all_variants(&nv);
  return nv;
}

}  // extern "C"
