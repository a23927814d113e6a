// fcm_chain.cpp -- FusePlanner over a chain of DW and PW layers (Sec. IV): every run of
// adjacent layers that forms a module (DW->PW, PW->DW, PW->PW, PW->DW->PW) or a single
// layer is planned with the module planner, and dynamic programming over the chain picks
// the partition into kernels of least total cost.
#include <algorithm>
#include <cstring>
#include <vector>

#include "fcm_host.h"

namespace fcm {

int op_layers(int op) {
  switch (op) {
    case FCM_OP_DW:
    case FCM_OP_PW: return 1;
    case FCM_OP_PW_DW_PW: return 3;
    default: return 2;
  }
}

// Layer kinds of each module, in execution order.
static bool op_matches(const fcm_chain_desc* c, int first, int op) {
  static const int kinds[6][3] = {{FCM_LAYER_DW, FCM_LAYER_PW, -1},  // DW_PW
                                  {FCM_LAYER_PW, FCM_LAYER_DW, -1},  // PW_DW
                                  {FCM_LAYER_PW, FCM_LAYER_DW, FCM_LAYER_PW},
                                  {FCM_LAYER_DW, -1, -1},
                                  {FCM_LAYER_PW, -1, -1},
                                  {FCM_LAYER_PW, FCM_LAYER_PW, -1}};
  const int n = op_layers(op);
  if (first < 0 || first + n > c->num_layers) return false;
  for (int i = 0; i < n; ++i)
    if (c->layers[first + i].kind != kinds[op][i]) return false;
  return true;
}

fcm_status chain_shapes(const fcm_chain_desc* c, int* h, int* w, int* ch) {
  if (!c) return fail(FCM_EINVAL, "chain is NULL");
  if (c->num_layers < 1 || c->num_layers > FCM_CHAIN_MAX_LAYERS)
    return fail(FCM_EINVAL, "chain: num_layers must be in [1, FCM_CHAIN_MAX_LAYERS]");
  if (c->n <= 0 || c->h <= 0 || c->w <= 0 || c->c <= 0) return fail(FCM_EINVAL, "chain: n, h, w, c must be positive");
  h[0] = c->h;
  w[0] = c->w;
  ch[0] = c->c;
  for (int i = 0; i < c->num_layers; ++i) {
    const fcm_layer& L = c->layers[i];
    if (L.kind == FCM_LAYER_PW) {
      if (L.c_out <= 0) return fail(FCM_EINVAL, "chain: a PW layer needs c_out > 0");
      h[i + 1] = h[i];
      w[i + 1] = w[i];
      ch[i + 1] = L.c_out;
    } else if (L.kind == FCM_LAYER_DW) {
      if (L.k <= 0 || L.stride <= 0 || L.pad < 0 || h[i] + 2 * L.pad < L.k || w[i] + 2 * L.pad < L.k)
        return fail(FCM_EINVAL, "chain: DW layer geometry leaves no output");
      h[i + 1] = (h[i] + 2 * L.pad - L.k) / L.stride + 1;
      w[i + 1] = (w[i] + 2 * L.pad - L.k) / L.stride + 1;
      ch[i + 1] = ch[i];
    } else {
      return fail(FCM_EINVAL, "chain: unknown layer kind");
    }
  }
  return FCM_OK;
}

fcm_status chain_group_desc(const fcm_chain_desc* c, const int* h, const int* w, const int* ch, int first, int op,
                            fcm_desc* d) {
  if (op < FCM_OP_DW_PW || op > FCM_OP_PW_PW || !op_matches(c, first, op))
    return fail(FCM_EINVAL, "chain: the layers do not form this module");
  memset(d, 0, sizeof(*d));
  d->n = c->n;
  d->h = h[first];
  d->w = w[first];
  d->dtype = c->dtype;
  d->layout = c->layout;
  d->k = 1;
  d->stride = 1;
  d->pad = 0;
  const int n = op_layers(op);
  for (int i = 0; i < n; ++i) {
    const fcm_layer& L = c->layers[first + i];
    d->act[i] = L.act;
    d->rq[i] = L.rq;
    if (L.kind == FCM_LAYER_DW) {
      d->k = L.k;
      d->stride = L.stride;
      d->pad = L.pad;
    }
  }
  // int8: the group's input zero point is the chain's or the previous layer's output one
  d->zp_in = first == 0 ? c->zp_in : c->layers[first - 1].rq.zero_point;
  d->c_in = ch[first];
  switch (op) {
    case FCM_OP_DW:
      d->c_mid = d->c_out = ch[first];
      break;
    case FCM_OP_PW:
      d->c_mid = ch[first];
      d->c_out = ch[first + 1];
      break;
    case FCM_OP_DW_PW:
      d->c_mid = ch[first];
      d->c_out = ch[first + 2];
      break;
    case FCM_OP_PW_DW:
      d->c_mid = d->c_out = ch[first + 1];
      break;
    default:  // PW_PW, PW_DW_PW: intermediate = first layer's output
      d->c_mid = ch[first + 1];
      d->c_out = ch[first + n];
      break;
  }
  // a module's rq/act slots beyond its stages stay as given (ignored)
  return FCM_OK;
}

}  // namespace fcm

using namespace fcm;

extern "C" {

fcm_status fcm_chain_plan(const fcm_chain_desc* chain, int32_t objective, const fcm_hw_desc* hw,
                          fcm_chain_plan_t* out) {
  if (!out) return fail(FCM_EINVAL, "output chain plan is NULL");
  if (objective < FCM_CHAIN_BYTES || objective > FCM_CHAIN_UNFUSED) return fail(FCM_EINVAL, "unknown objective");
  std::vector<int> h(FCM_CHAIN_MAX_LAYERS + 1), w(FCM_CHAIN_MAX_LAYERS + 1), ch(FCM_CHAIN_MAX_LAYERS + 1);
  fcm_status st = chain_shapes(chain, h.data(), w.data(), ch.data());
  if (st != FCM_OK) return st;
  const fcm_hw_desc H = hw ? *hw : default_hw();
  const int n = chain->num_layers;

  // every candidate group: (first layer, op) -> plan and its costs
  struct Opt {
    int op;
    fcm_plan_t plan;
    double bytes, time;
  };
  std::vector<std::vector<Opt>> opts(n);
  static const int kOps[6] = {FCM_OP_DW, FCM_OP_PW, FCM_OP_DW_PW, FCM_OP_PW_DW, FCM_OP_PW_PW, FCM_OP_PW_DW_PW};
  for (int i = 0; i < n; ++i) {
    for (int op : kOps) {
      if (!op_matches(chain, i, op)) continue;
      const bool single = op == FCM_OP_DW || op == FCM_OP_PW;
      if (!single && objective == FCM_CHAIN_UNFUSED) continue;
      fcm_desc d;
      st = chain_group_desc(chain, h.data(), w.data(), ch.data(), i, op, &d);
      if (st != FCM_OK) return st;
      st = validate(op, &d);
      if (st == FCM_EINVAL) return st;  // an invalid layer is an error of the chain
      if (st != FCM_OK) {
        if (single) return st;  // a layer no kernel implements
        continue;               // a module no kernel implements: the layers stay apart
      }
      Opt o;
      o.op = op;
      // groups run with the chain's activation buffers only: plans without split workspace
      st = find_plan(op, &d, &H, &o.plan, kernel_set(op, &d), 0);
      if (st != FCM_OK) {
        if (single) return st;
        continue;
      }
      o.bytes = (double)o.plan.bytes_paper;
      o.time = plan_time_estimate(geometry(op, &d), o.plan, H);
      opts[i].push_back(o);
    }
  }
  // dynamic programming from the end: best[i] = least cost of layers i .. n-1; options at
  // a position are tried singles first and replaced only by a strictly smaller cost
  std::vector<double> best(n + 1, 0.0);
  std::vector<int> pick(n, -1);
  for (int i = n - 1; i >= 0; --i) {
    best[i] = -1.0;
    for (int k = 0; k < (int)opts[i].size(); ++k) {
      const Opt& o = opts[i][k];
      const double cst = (objective == FCM_CHAIN_TIME ? o.time : o.bytes) + best[i + op_layers(o.op)];
      if (best[i] < 0.0 || cst < best[i]) {
        best[i] = cst;
        pick[i] = k;
      }
    }
    if (pick[i] < 0) return fail(FCM_EUNSUPPORTED, "chain: a layer has no compiled kernel");
  }
  memset(out, 0, sizeof(*out));
  out->objective = objective;
  int g = 0;
  for (int i = 0; i < n;) {
    const Opt& o = opts[i][pick[i]];
    out->first[g] = i;
    out->op[g] = o.op;
    out->plan[g] = o.plan;
    out->bytes_paper += o.plan.bytes_paper;
    out->time_est += o.time;
    const int len = op_layers(o.op);
    if (len > 1) out->fused_layers += len;
    i += len;
    if (i < n) {
      const int64_t e = chain->dtype == FCM_F32 ? 4 : (chain->dtype == FCM_BF16 ? 2 : 1);
      out->act_bytes_max = std::max(out->act_bytes_max, (int64_t)chain->n * h[i] * w[i] * ch[i] * e);
    }
    ++g;
  }
  out->num_groups = g;
  for (int i = 0; i < n; ++i)
    for (const Opt& o : opts[i])
      if (o.op == FCM_OP_DW || o.op == FCM_OP_PW) {
        out->bytes_lbl_paper += o.plan.bytes_paper;
        out->time_lbl_est += o.time;
      }
  return FCM_OK;
}

int64_t fcm_chain_workspace_bytes(const fcm_chain_plan_t* plan) {
  if (!plan || plan->num_groups <= 1) return 0;
  return 2 * ((plan->act_bytes_max + 255) / 256 * 256);
}

}  // extern "C"
