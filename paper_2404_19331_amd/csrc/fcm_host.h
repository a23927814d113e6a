// fcm_host.h -- host-side internals shared by the planner and the C ABI.
#pragma once

#include <stdint.h>

#include <string>

#include "fcm.h"
#include "fcm_internal.h"

namespace fcm {

// Record a failure message for fcm_last_error() and return the status.
fcm_status fail(fcm_status st, const std::string& msg);

// Kernel sets a descriptor may run on: the first-generation kernels always; with
// KSET_DMA every kernel; with KSET_REG only (zero points) also the int8 persistent
// kernels and the PW->PW register kernel's instances of at most
// kZpMaxTiles output tiles.
// KSET_PC (per-channel requantisation): the first-generation kernels and the int8
// persistent kernels only.
enum { KSET_FIRST = 0, KSET_DMA = 1, KSET_REG = 2, KSET_ALL = 3, KSET_PC = 4 };
// The set an int8 descriptor's features allow: per-channel requantisation -> KSET_PC;
// zero points -> KSET_REG; else all.
int kernel_set(int op, const fcm_desc* d);
// Whether an int8 descriptor has a nonzero zero point (zp) or per-channel requantisation
// (pc) in any stage of module `op` (0 and 0 for float types).
void int8_features(int op, const fcm_desc* d, int* zp, int* pc);
// Whether compiled variant `variant` belongs to kernel set `kset`.
bool variant_in_set(int variant, int kset);

// Argument checks common to fcm_plan and every launch entry point.
fcm_status validate(int op, const fcm_desc* d);

// Geometry derived from a descriptor for one module.
struct Geom {
  int op, family;
  int n, h, w;          // input
  int ci, cm, co;       // input / intermediate / output channels of the module
  int k, s, pad;        // depthwise (1, 1, 0 for the pointwise layer)
  int ho, wo;           // output
  int dtype, elt;
  int layout;
  int zp;               // int8 with a nonzero zero point in any stage (time models)
  int pc;               // int8 with per-channel requantisation in any stage
};
Geom geometry(int op, const fcm_desc* d);

// Fill every derived field of a plan whose op/tile/c_block/co_block/variant are set.
// Returns FCM_EUNSUPPORTED if the variant cannot implement the tiling.
fcm_status evaluate_plan(const Geom& g, const fcm_desc* d, const fcm_hw_desc& hw, fcm_plan_t* p);

// Search (cached) over the variants of kernel set kset. plan_out is fully filled on
// success.
// ws_max: the largest caller workspace a plan may need (split plans of the persistent
// kernels keep their partial sums there); plans needing more are not considered.
fcm_status find_plan(int op, const fcm_desc* d, const fcm_hw_desc* hw, fcm_plan_t* plan_out, int kset = KSET_ALL,
                     int64_t ws_max = INT64_MAX);

// Device workspace bytes a (fully evaluated) plan needs: the partial sums of a split plan,
// 0 for every other plan.
// Up to max_count plans for the shape: the planner's choice first, then each kernel
// variant's best plan by the time models, then the rest, fastest first.
fcm_status find_candidates(int op, const fcm_desc* d, const fcm_hw_desc* hw, int kset, int64_t ws_max,
                           fcm_plan_t* out, int max_count, int* count);
int64_t plan_workspace_bytes(const Geom& g, const fcm_plan_t& p);

// Whether a compiled variant stages through LDS-DMA (needs 16-byte aligned tensors).
bool variant_needs_alignment(int variant);

fcm_hw_desc default_hw();

// Estimated seconds of a plan's launch: the fitted time model of its kernel family where
// there is one (persistent DW->PW / PW / DW kernels, PW->PW register kernel), else its
// bytes at the HBM rate plus a launch.
double plan_time_estimate(const Geom& g, const fcm_plan_t& p, const fcm_hw_desc& hw);

// Chains: input shape of every layer (h[i], w[i], c[i] for layer i; index num_layers is
// the chain output) after checking the chain's sizes and geometry.
fcm_status chain_shapes(const fcm_chain_desc* c, int* h, int* w, int* ch);

// Descriptor of the module `op` over the chain's layers first, first+1, ... (their count
// follows from op), or FCM_EINVAL if those layers do not form that module.
fcm_status chain_group_desc(const fcm_chain_desc* c, const int* h, const int* w, const int* ch, int first, int op,
                            fcm_desc* d);

// Number of layers a module spans.
int op_layers(int op);

// Launch module `op` (validation, planning, launch) with an optional caller workspace for
// split plans: the body of every launch entry point. w / b: the module's weights and
// biases in execution order (unused ones NULL).
fcm_status launch_module(int op, const fcm_desc* d, const void* x, const void* const* w, const void* const* b,
                         void* y, const fcm_plan_t* plan, void* ws, int64_t ws_bytes, void* stream);

}  // namespace fcm
