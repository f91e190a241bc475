// Host-side launchers of the HIP kernels. Arguments are validated by the
// C-ABI layer before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "base.h"

namespace base {

// rows: null, or output row i reads row rows[i] of H (h_rows rows).
hipError_t launch_affinity_bf16(const uint16_t *H, const int32_t *rows, int64_t h_rows,
                                const uint16_t *W, float *S, int64_t T, int64_t E, int64_t d,
                                hipStream_t stream);
hipError_t launch_affinity_f32(const float *H, const int32_t *rows, int64_t h_rows,
                               const float *W, float *S, int64_t T, int64_t E, int64_t d,
                               hipStream_t stream);

// B problems of T rows; shuffle: null or the [B*T] index composed after perm.
hipError_t launch_permute(const void *in, const int32_t *perm, const int32_t *shuffle,
                          void *out, int64_t B, int64_t T, int64_t row_bytes, int inverse,
                          hipStream_t stream);

struct AssignParams {
    int64_t T, E, C;
    bool integer;         // int16 scores, int64 arithmetic
    int64_t scale;        // integer mode: K; float mode: 1
    double eps_final;     // score units (float) / scaled units (integer)
    double eps_initial;   // <= 0: derived from the score range on the device
    double eps_factor;
    int32_t max_rounds;
    uint32_t flags;
    const void *warm_prices;   // non-null: initial prices ([B][E], the prices output layout)
};

// Round bound of a solve whose caller sets none (max_rounds <= 0).
constexpr int32_t kDefaultMaxRounds = 4000000;

// Device-side solver state and statistics, at the head of the workspace.
struct SolveCtrl {
    int32_t active_count[2];
    int32_t cur;            // which active list the next round reads
    int32_t all_active;     // 1: every token is active (first round of a phase)
    int32_t phase;          // phases started
    int32_t rounds;         // rounds run over all phases
    int32_t done;           // 1 once the last phase has finished
    int32_t overflow;       // a bid left the key's range
    int32_t not_converged;  // max_rounds reached
    int32_t fell_back;
    int32_t last_phase;     // the current phase runs at eps_final
    int32_t blocks_done;    // last-block counter of the wide update kernel
    uint32_t smax_ord, smin_ord;   // score range (order-preserving images)
    int32_t unconverged_experts;
    int32_t pad0;
    unsigned long long bids;
    double eps;             // epsilon of the current phase (score or scaled units)
    double eps_final_eff;
    int32_t internal_error; // a device-side consistency check failed
    int32_t pad2;
    unsigned long long engine_bids;   // bids placed inside the single-workgroup engine
    double dual_gap;        // D(p) - objective after the solve (when statistics are asked for)
    int32_t certified;      // 1: stopped after a phase whose duality gap met T eps_final
    int32_t skip_check;     // 1: the current phase ended before its last tokens were placed
    double check_gap;       // duality gap measured after the last phase (0: not measured)
    int64_t scale;          // integer mode: K (scores are scaled by it); float mode: 1
    int32_t integer;        // 1: integer mode
    int32_t augmentations;  // shortest augmenting paths run over all phases
    int32_t early_ok;       // 1: the current phase may end early (its epsilon is large)
    int32_t pad4;
};

// The validated assign call shared by base_assign, base_assign_batched and
// base_assign_noalloc (arguments and result as base_assign_batched).
int assign_entry(const void *S, int s_dtype, int64_t B, int64_t T, int64_t E,
                 const base_assign_opts *opts, int32_t *assign, int32_t *perm, void *prices,
                 void *workspace, size_t workspace_bytes, base_assign_stats *stats, void *stream);

// Status and statistics of B problems from their control blocks (aggregated
// as documented for base_assign_stats). Returns a base_status code.
int aggregate_stats(const SolveCtrl *cs, int64_t B, int64_t E, bool with_gap, void *stats_out);

size_t assign_workspace_size(int64_t T, int64_t E);

// Enqueues the whole solve of B independent problems of T x E scores
// (scores, outputs and workspaces laid out problem after problem).
hipError_t launch_assign(const void *S, const AssignParams &p, int64_t B, int32_t *assign,
                         int32_t *perm, void *prices_out, void *workspace, hipStream_t stream);

// Reads the B control blocks back (synchronises the stream).
hipError_t read_assign_stats(const void *workspace, int64_t T, int64_t E, int64_t B,
                             SolveCtrl *out, hipStream_t stream);

// Test-time routing (argmax per token, stable counting sort) and the gated
// residual of Eq. 1 with its gradient (gate.hip).
size_t greedy_workspace_size(int64_t T, int64_t E);
hipError_t launch_greedy(const float *S, int64_t T, int64_t E, int32_t *assign, int32_t *perm,
                         int32_t *offsets, void *workspace, hipStream_t s);
// B problems of T tokens; shuffle: null or the [B*T] worker -> token index.
hipError_t launch_gate_combine(const void *F, const void *H, const float *S,
                               const int32_t *assign, const int32_t *perm,
                               const int32_t *shuffle, void *Y, int64_t B, int64_t T, int64_t E,
                               int64_t d, int bf16, hipStream_t s);
hipError_t launch_gate_backward(const void *dY, const void *F, const void *H, const void *W,
                                const float *S, const int32_t *assign, const int32_t *perm,
                                const int32_t *offsets, void *dH, void *dF, float *dW, float *dS,
                                int64_t T, int64_t E, int64_t d, int bf16, hipStream_t s);

// Event timing of the engine kernel's launches (measurement support).
hipError_t timing_enable(int32_t capacity);
hipError_t timing_read(int64_t *launches, double *total_ms);

// Scans S for NaN/Inf (synchronous). *bad is set to 1 when one is found.
// Scans n scores for NaN/Inf (synchronous), using the workspace of one
// T x E problem. *bad is set to 1 when one is found.
hipError_t check_scores_finite(const float *S, int64_t n, int64_t T, int64_t E, void *workspace,
                               int *bad, hipStream_t stream);

}  // namespace base
