/*
 * ardit_control.h -- the playout-slack controller of libardit (host code).
 *
 * The decisions that pick which stream's chunk runs next, where, and at which
 * fidelity (paper, Sections 3-5): service credit, urgency tiers and dispatch
 * order, credit-aware eviction, re-homing, the elastic-SP donor, admission, and
 * Bi-Modal Pareto Routing over the profiled fidelity configurations.  Every
 * call is plain host computation on caller-owned host arrays: no HIP call, no
 * allocation that outlives the call, no state kept between calls.  Times are
 * milliseconds (double).  Status codes are ardit_status (ardit.h); on a
 * failed check nothing is written.
 *
 * Readings where the paper leaves a choice open (each call states its own):
 * the BMPR budget of a stream is the slack left when its next chunk can start,
 * P - R; ties are broken as stated per call.
 */
#ifndef ARDIT_CONTROL_H
#define ARDIT_CONTROL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* One fidelity configuration (Section 2.1 knobs; Appendix A space:
 * S in {2,3,4}, rho in {0,.6,.7,.8,.9}, W in {1,3,7}, Q in {FP16, FP8}) with
 * its profiled latency per chunk and quality score (higher is better). */
typedef struct {
  int32_t steps;       /* S */
  float sparsity;      /* rho */
  int32_t window;      /* W, prior chunks kept */
  int32_t quant;       /* ardit_quant */
  double latency_ms;   /* L: profiled generation time of one chunk */
  double quality;      /* Q */
} ardit_fidelity;

typedef enum { ARDIT_URGENT = 0, ARDIT_NORMAL = 1, ARDIT_RELAXED = 2 } ardit_tier;
typedef enum { ARDIT_BMPR_QUALITY = 0, ARDIT_BMPR_SPEED_RECOVERY = 1 } ardit_bmpr_mode;

/* Offline construction (Section 5.2; Appendix A): the non-dominated
 * configurations (j dominates i when L_j <= L_i and Q_j >= Q_i with one
 * inequality strict; identical points are both kept), written to frontier[]
 * (room for n) in order of latency ascending, then quality descending, then
 * index; *n_frontier their count; *q_floor the median quality over all n
 * configurations (mean of the middle two for even n).  EINVAL on n < 1 or a
 * non-finite latency or quality. */
int ardit_pareto_frontier(int32_t n, const ardit_fidelity* cfgs, int32_t* frontier,
                          int32_t* n_frontier, double* q_floor);

/* Online selection (Section 5.2) for a budget B: quality mode, the frontier
 * point of highest quality with L <= B and Q >= q_floor (ties: lower latency,
 * then lower index); if there is none, speed-recovery mode, the frontier point
 * of lowest latency with Q >= q_floor (ties: higher quality, then lower index).
 * Writes the configuration index and the mode.  ECAPACITY when no frontier
 * point reaches the floor (a frontier built from the same configurations
 * always holds the best one, which does). */
int ardit_bmpr_select(int32_t n_cfgs, const ardit_fidelity* cfgs, int32_t n_frontier,
                      const int32_t* frontier, double q_floor, double budget_ms, int32_t* cfg,
                      int32_t* mode);

/* Per-stream state the controller reads at a tick. */
typedef struct {
  int32_t worker;            /* current home worker */
  int32_t sp_donor;          /* donor worker of the stream's SP2 group, -1 when none */
  double slack_ms;           /* P: playable buffer left */
  double remaining_ms;       /* R: estimated time to finish the running chunk, 0 if not running */
  double cooldown_until_ms;  /* re-homing cooldown end (controller clock), -inf when none */
} ardit_stream_state;

typedef struct {
  int32_t n_workers;
  int32_t gpus_per_node;     /* workers w and w' share a node when w / g == w' / g */
  int32_t cap_send;          /* migrations out of one worker per tick (2) */
  int32_t cap_recv;          /* migrations into one worker per tick (1) */
  double cooldown_ms;        /* after a migration (60000) */
  double now_ms;             /* controller clock */
} ardit_ctl_params;

/* What a tick decides for one stream. */
typedef struct {
  int32_t cfg;               /* next chunk's configuration (BMPR with budget P - R) */
  int32_t mode;              /* ardit_bmpr_mode */
  int32_t tier;              /* ardit_tier under cfg */
  int32_t queue_pos;         /* 0-based position in its worker's dispatch order */
  int32_t rehome_to;         /* destination worker planned this tick, -1 */
  int32_t sp_donor;          /* donor after this tick, -1 */
  double credit_ms;          /* C = P - (R + L_cfg) */
  double cooldown_until_ms;  /* updated when the stream is re-homed */
} ardit_stream_decision;

/* One control tick (Appendix C.1 order):
 *  1. per stream: cfg by BMPR with budget P - R; credit C = P - (R + L_cfg);
 *     tier URGENT when C < 2 L_cfg, RELAXED when C > 4 L_cfg, else NORMAL
 *     (Sections 3.1, 4.1);
 *  2. dispatch order per worker: ascending credit, then stream index;
 *  3. re-homing (Section 4.2 and its algorithm; Appendix C.2): senders are
 *     workers holding at least two URGENT streams, most URGENT streams first
 *     (then lower id); receivers are workers with no URGENT or NORMAL stream
 *     (idle ones included), tried same-node first, then by id; while the
 *     sender has sent fewer than cap_send and the receiver received fewer
 *     than cap_recv, the sender's lowest-credit URGENT stream that is not in
 *     cooldown, not in an SP2 group and not yet moved goes to that receiver
 *     and enters cooldown until now + cooldown_ms;
 *  4. elastic SP (Section 4.3; Appendix C.3): a stream keeps its donor until
 *     C >= 2 L_cfg (NORMAL), then releases it; each stream with C < 0 that has
 *     no donor and is not being re-homed, in ascending credit order, borrows
 *     the highest-credit worker on its own node (a worker's credit: the lowest
 *     of its streams', +inf when idle; ties to the lower id) that has no
 *     URGENT or NORMAL stream, is not its own worker, is not lending and did
 *     not receive a migration this tick; none is borrowed when there is none.
 * streams / out: n_streams entries.  EINVAL on a malformed argument (worker
 * or donor out of range, non-finite slack or remaining time, empty
 * frontier). */
int ardit_control_tick(const ardit_ctl_params* params, int32_t n_cfgs,
                       const ardit_fidelity* cfgs, int32_t n_frontier, const int32_t* frontier,
                       double q_floor, int32_t n_streams, const ardit_stream_state* streams,
                       ardit_stream_decision* out);

/* Credit-aware eviction (Section 4.1): to make room for need_pages of stream
 * `requester` when free_pages are free, evict resident streams other than the
 * requester (resident_pages[i] > 0) in order of credit descending (ties: the
 * higher index first) until the pages fit.  Writes the evicted indices in
 * order to evict[] (room for n) and their count.  ECAPACITY (nothing written)
 * when evicting every other resident stream would still leave too few. */
int ardit_evict_for(int32_t n, const double* credits, const int32_t* resident_pages,
                    int32_t requester, int64_t free_pages, int64_t need_pages, int32_t* evict,
                    int32_t* n_evict);

/* Admission (Section 3.3): the home worker is the one with the fewest
 * streams (lowest id on ties); the initial slack (the time-to-first-chunk
 * budget) is 4x the estimated first-chunk time. */
int ardit_admit(int32_t n_workers, const int32_t* streams_per_worker, double first_chunk_ms,
                int32_t* home, double* slack_ms);

#ifdef __cplusplus
}
#endif

#endif /* ARDIT_CONTROL_H */
