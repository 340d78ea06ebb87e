/*
 * ardit_control.h -- the playout-slack controller of libardit (host code).
 *
 * The decisions that pick which stream's chunk runs next and at which fidelity
 * (paper, Sections 3-5): service credit, urgency tiers and dispatch order, and
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
  int32_t worker;            /* home worker (0 .. n_workers - 1) */
  double slack_ms;           /* P: playable buffer left */
  double remaining_ms;       /* R: estimated time to finish the running chunk, 0 if not running */
} ardit_stream_state;

/* What a tick decides for one stream. */
typedef struct {
  int32_t cfg;               /* next chunk's configuration (BMPR with budget P - R) */
  int32_t mode;              /* ardit_bmpr_mode */
  int32_t tier;              /* ardit_tier under cfg */
  int32_t queue_pos;         /* 0-based position in its worker's dispatch order */
  double credit_ms;          /* C = P - (R + L_cfg) */
} ardit_stream_decision;

/* One control tick over the streams of n_workers workers (Appendix C.1 order,
 * its first two decisions):
 *  1. per stream: cfg by BMPR with budget P - R; credit C = P - (R + L_cfg)
 *     (Section 3.1); tier URGENT when C < 2 L_cfg, RELAXED when C > 4 L_cfg,
 *     else NORMAL (Section 4.1);
 *  2. dispatch order per worker: ascending credit, then stream index
 *     (Section 4.1, credit-ordered queues).
 * streams / out: n_streams entries.  EINVAL on a malformed argument (worker
 * out of range, non-finite slack or remaining time, empty frontier). */
int ardit_control_tick(int32_t n_workers, int32_t n_cfgs, const ardit_fidelity* cfgs,
                       int32_t n_frontier, const int32_t* frontier, double q_floor,
                       int32_t n_streams, const ardit_stream_state* streams,
                       ardit_stream_decision* out);

#ifdef __cplusplus
}
#endif

#endif /* ARDIT_CONTROL_H */
