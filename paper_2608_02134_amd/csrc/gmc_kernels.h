// Host-side launchers of the GMC kernels (one per stage).  All enqueue on
// `st` and never synchronise.
#pragma once

#include <hip/hip_runtime.h>

#include "gmc_internal.h"

namespace gmc {

// Stage ids of the measurement timer (see gmc_timing_enable in gmc.h).
enum Stage {
  kStProbe = 0, kStLogits, kStHeads, kStAppearance, kStSpatial, kStCov, kStGains, kStResp,
  kStObjective, kStAssign, kStTransport, kStInit, kStSelect, kNumStages
};
// Records a hipEvent on `st` opening (begin) or closing a stage span when
// timing is enabled; a no-op otherwise.
void timer_mark(int stage, bool begin, hipStream_t st);

// Squared row norms of the visual states (every later stage reads them).
// call_tag != 0: every block also tags itself done with it for the gate.
hipError_t launch_rownorm(const Shape& sh, const Ws& ws, const void* hidden, int call_tag, hipStream_t st);

// One block that returns once every row-norm block carries call_tag.
hipError_t launch_bank_gate(const Shape& sh, const Ws& ws, int call_tag, hipStream_t st);

// The inputs of one message view: its states, queries, keys, folded value
// probe (and bias) and optional nonvisual log-sum-exp.
struct MsgView {
  const void* hidden;
  const void* text_q;
  const void* vis_k;
  const void* probe;
  const float* probe_bias;
  const float* nonvis_lse;
};

// Value probe, mass coordinate, native slice of every message view (views[0]
// the current one, sh.nviews in all), head weights over the views' patterns,
// grounded row weights and the current view's energy (after launch_rownorm).
// With bank_flag set (T > 0), the last kernel also waits until the flag
// reads 1.
hipError_t launch_message(const Shape& sh, const Params& pr, const Ws& ws, const MsgView* views,
                          float* trace_omega, const int* bank_flag, hipStream_t st);

// Sets *flag = 1 once the work before it on st has finished.
hipError_t launch_bank_signal(int* flag, hipStream_t st);

// Appearance (exact or bounded) and spatial banks with their row weights.
hipError_t launch_banks(const Shape& sh, const Params& pr, const Ws& ws, const void* hidden,
                        const void* app_proj, const int32_t* pos3d, hipStream_t st);

// All selection rounds, then the final coverage and objective values.
// *support_ready reports that the support list and slots were written too.
// `so` receives each round's pool, batch, gains and pool scores (any may be
// NULL).
hipError_t launch_selection(const Shape& sh, const Params& pr, const Ws& ws, const SelOut& so, hipStream_t st,
                            bool* support_ready);

// Certificate of the selection rounds from the exported per-round pools,
// batches, gains and scores (all of `so` set; sh.rounds <= ws.cert_rounds).
hipError_t launch_certificate(const Shape& sh, const Ws& ws, const SelOut& so, hipStream_t st);

// Debug scan for non-finite client energies, row weights and outputs.
hipError_t launch_finite_scan(const Shape& sh, const Ws& ws, const void* out_hidden, hipStream_t st);

// Multi-image calls: clamped image ids and per-image token counts.
hipError_t launch_image_prep(const Shape& sh, const Ws& ws, const int32_t* image_id, hipStream_t st);

// Multi-image calls: S_0, the largest singleton gain F({i}) of every image
// (ties to the lower index), marked selected, recorded first in the support
// order, and the coverage b_m(S_0).
hipError_t launch_image_seeds(const Shape& sh, const Ws& ws, hipStream_t st);

// Scratch of the realisation audit, carved from the context workspace.
struct AudWs {
  float* A;      // [B][N][mg1]   Full attention, token-major
  float* Y;      // [B][mg1][dh]  Full messages
  float* lse;    // [B][mg1]      Full log-sum-exp (with the nonvisual part)
  float* Mt;     // [B][K][mg1]   grouped Full mass, carrier-major
  int* off;      // [B][K + 1]    member list offsets per carrier
  int* mem;      // [B][N]        members, ascending within a carrier
  int* cur;      // [B][K]        placement cursors
  float* rowst;  // [B][mg1][kAuditRow] per-client statistics
};

// Signed-message realisation audit (Full and compact native attention,
// grouped mass, decomposition terms, weighted e_M / alpha / kappa).
hipError_t launch_audit(const Shape& sh, const AudWs& aw, const void* text_q, const void* vis_k,
                        const void* vis_v, const void* comp_k, const void* comp_v, const int32_t* carrier,
                        const float* weights, const float* nonvis_lse, float* rows_out, float* vec_out, float* out,
                        hipStream_t st);

// Clears the device status words of problems [0, nprob).
hipError_t launch_clear_status(const Ws& ws, int nprob, hipStream_t st);

// Support list, selected-cosine gaps, separability gate, assignment.
hipError_t launch_assignment(const Shape& sh, const Params& pr, const Ws& ws, const void* hidden,
                             bool support_ready, int32_t* trace_assign, hipStream_t st);

// Population weights, weighted centroids, RMS restoration, compaction.
hipError_t launch_transport(const Shape& sh, const Params& pr, const Ws& ws, const void* hidden,
                            const int32_t* pos3d, void* out_hidden, int32_t* out_pos,
                            int32_t* out_idx, hipStream_t st);

// K = N: copy inputs to outputs.
hipError_t launch_identity(const Shape& sh, const void* hidden, const int32_t* pos3d,
                           void* out_hidden, int32_t* out_pos, int32_t* out_idx, hipStream_t st);

// Sequence compaction after pruning: index map, inverse map, boundary rows
// and position ids (row_chunks = row bytes / 16; NULL outputs are skipped).
hipError_t launch_compact_sequence(int B, int L, int v0, int N, int K, const int32_t* out_idx, int32_t* iota,
                                   int32_t* keep, const void* seq_rows, const void* vis_rows, void* out_rows,
                                   int row_chunks, const int32_t* seq_pos, int32_t* out_pos, hipStream_t st);

// Row gather of up to kMaxGather tensors at the retained positions.
hipError_t launch_gather_rows(int n_tensors, const void* const* src, void* const* dst, int n_seq, int spk, int L,
                              int L2, int row_chunks, const int32_t* keep, hipStream_t st);

// Debug exports: pre-weighted client matrix and per-problem statistics.
hipError_t launch_trace_exports(const Shape& sh, const Ws& ws, float* trace_client,
                                float* trace_stats, float* trace_ebar, hipStream_t st);

}  // namespace gmc
