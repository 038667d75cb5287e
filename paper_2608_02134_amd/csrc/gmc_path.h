// The host side of one pruning call, shared by the context entry points and
// the static-scratch entry point: shape resolution, argument checks, the
// workspace plan and the launch sequence.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gmc.h"
#include "gmc_internal.h"

namespace gmc {

// Capacities a call is checked against.
struct Limits {
  int B, N, T, K, H, I;   // H: historical message views, I: images
};

// Streams of one call: everything runs on `st`; with `side` set the bank
// kernels run there, forked by the row-norm gate (call_tag != 0) or by the
// `fork` event, and joined by a device flag (T > 0) or the `join` event.
struct PathStreams {
  hipStream_t st;
  hipStream_t side;
  int call_tag;
  hipEvent_t fork, join;
};

// Records the message gmc_last_error() returns; returns code.
int set_error(int code, const char* fmt, ...);

// Validates a configuration (gmc_init's checks).
int check_config(const gmc_config* cfg);

// The frozen settings of a configuration, as the kernels take them.
Params params_of(const gmc_config& cfg);

// Carves the workspace of a configuration's capacities out of `base` (or
// only sizes it when base is NULL); returns its bytes.
size_t carve_workspace(const gmc_config& cfg, char* base, Ws* ws);

// Resolves a call's shape against the limits.
int resolve_shape(const gmc_config& g, const Limits& cap, int64_t B, int64_t N, int64_t T, int64_t K_req,
                  Shape* out, int64_t n_hist = 0, int64_t n_images = 1);

// Null pointers and overlapping outputs (historical views: hist[0, n_hist)).
int check_tensors(const Shape& s, const void* hidden, const void* text_q, const void* vis_k, const int32_t* pos3d,
                  const void* out_hidden, const int32_t* out_pos, const int32_t* out_idx,
                  const gmc_view* hist = nullptr);

// Enqueues the whole operator (or the identity copy when K = N).
// Historical views: hist[0, s.nviews - 1).
int enqueue_prune(const gmc_config& cfg, const Params& pr, const Ws& ws, const Shape& s, const PathStreams& ps,
                  int diag, const void* hidden, const void* text_q, const void* vis_k, const int32_t* pos3d,
                  void* out_hidden, int32_t* out_pos, int32_t* out_idx, const float* nonvis_lse,
                  const gmc_trace& tr, bool* cert_done, const gmc_view* hist = nullptr,
                  const int32_t* image_id = nullptr);

}  // namespace gmc
