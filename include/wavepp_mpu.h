/*
 * wavepp_mpu.h -- C ABI of the Maximum Pipeline Utilization (MPU) wave planner in
 * libwavepp_attn.so: it chooses each wave's token budget and packs the admitted requests' chunks
 * into waves, producing the spans (request, starting token, length) that the chunked-prefill
 * entry points consume.  Host only: no HIP call.
 *
 * Behaviour (Design of WavePP, "Pipeline Scheduling"):
 *   - P pipeline stages, an execution ring of R = 2P waves, a target of S = R + (F - 1) P waves.
 *   - Budgets b_0 = M, b_{j+1} = max(b_min, alignDown_B(b_j / 2)) (Eq. 6).
 *   - W = unscheduled suffix tokens of the admitted requests plus each one's most recently
 *     committed chunk while its wave is in the ring (count_inflight = 1); pieces are those
 *     suffixes and chunks; n(b) = max(W / b, N_{>b/2}) (Eq. 7), evaluated exactly in integers.
 *   - The largest budget with n(b) >= S is the target, b_min if none; once a budget supplies R
 *     waves, halving it is refused if the pieces it would newly split exceed split_permille / 1000
 *     of W (the paper uses 12.5 %).
 *   - The first decision takes its target.  Later, a target two or more halvings above the
 *     current budget is adopted at once; one halving above, after R/2 decisions in a row; a
 *     smaller one after R decisions in a row and only if the current budget is at least a full
 *     wave short of S (n(b) <= S - 1).
 *   - Packing is first-come-first-served (admission order), one chunk per request, at most
 *     max_lanes requests per wave, and stops at the first request it cannot place; a fragment of
 *     a request that does not fit whole is not put into a leftover space smaller than
 *     max(b_min, b / 2).
 *   - While the ring is busy, a wave holding a single request below half the budget is held back
 *     for one planning iteration when the caller reports a request in admission.
 *   - The caller commits the spans the scheduler actually accepted (possibly shorter, or fewer);
 *     positions advance only by those.  A span that does not start at its request's position is
 *     rejected with WAVEPP_EPOSITION.
 *
 * Ownership: the planner is a host object owned by the library until wavepp_mpu_destroy.  It is
 * not thread-safe: one thread (the scheduling rank) drives it.
 * Errors: wavepp_status codes (wavepp_attn.h), details in wavepp_last_error().
 */
#ifndef WAVEPP_MPU_H
#define WAVEPP_MPU_H

#include "wavepp_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t max_budget;       /* M, a multiple of block */
  int32_t min_budget;       /* b_min, a multiple of block, block <= b_min <= M */
  int32_t block;            /* B */
  int32_t stages;           /* P >= 1 */
  int32_t fills;            /* F >= 1 */
  int32_t max_lanes;        /* requests per wave >= 1 */
  int32_t split_permille;   /* 0..1000; the paper's 12.5 % is 125 */
  int32_t count_inflight;   /* 1: W and the pieces include in-flight chunks; 0: unscheduled tokens only */
} wavepp_mpu_config;

typedef struct {
  int32_t request;
  int32_t start;
  int32_t length;
} wavepp_span;

typedef struct {
  int64_t work;             /* W at this moment */
  int32_t budget;           /* budget of the last decision, 0 before the first */
  int32_t ring;             /* waves in the ring */
  int32_t requests;         /* admitted requests still tracked */
  int32_t up_count;
  int32_t down_count;
} wavepp_mpu_state;

typedef struct wavepp_mpu_s wavepp_mpu_t;

/* Write the budget ladder of Eq. 6 (largest first); returns its length, or a negative status.
 * Writes min(capacity, length) entries. */
int wavepp_mpu_budget_ladder(const wavepp_mpu_config* config, int32_t* out, int32_t capacity);

int wavepp_mpu_create(const wavepp_mpu_config* config, wavepp_mpu_t** out);

/* Admit request `request` whose uncached suffix is tokens [start, end).  Ids must be unique among
 * the tracked requests; admission order is the packing order. */
int wavepp_mpu_admit(wavepp_mpu_t* planner, int32_t request, int32_t start, int32_t end);

/* One planning decision.  Writes up to max_lanes spans (capacity must be >= max_lanes) and the
 * budget used; returns the number of spans, 0 when nothing is to be scheduled now (ring full, no
 * work, or a lone small wave held back), or a negative status. */
int wavepp_mpu_plan(wavepp_mpu_t* planner, int32_t admission_pending, wavepp_span* spans, int32_t capacity,
                    int32_t* budget);

/* The scheduler accepted these spans as one wave entering the ring.  Returns the wave's serial
 * (>= 1) or a negative status; on error nothing changes. */
int wavepp_mpu_commit(wavepp_mpu_t* planner, const wavepp_span* spans, int32_t n);

/* The oldest wave in the ring left the last stage. */
int wavepp_mpu_retire(wavepp_mpu_t* planner);

int wavepp_mpu_get_state(const wavepp_mpu_t* planner, wavepp_mpu_state* state);

void wavepp_mpu_destroy(wavepp_mpu_t* planner);

#ifdef __cplusplus
}
#endif

#endif /* WAVEPP_MPU_H */
