/*
 * vpp_sched.h -- discrete-event model of chunked-prefill pipeline schedules on
 * two pipeline ranks, fed by measured per-chunk latencies.
 *
 * The schedules (paper: "VPP: Virtual Pipeline Parallelism for Efficient
 * Chunked Prefill in Long-Context LLM Inference"):
 *
 *   CPP (sections 2.4 and 4): the layers are split into two physical stages,
 *   rank 0 then rank 1; every chunk runs stage 0 on rank 0, then stage 1 on
 *   rank 1, in chunk order.
 *
 *   VPP (section 5.1): the layers are split into four virtual stages s0..s3;
 *   s0 and s3 run on rank 0, s1 and s2 on rank 1, and every chunk follows the
 *   V-shaped route s0 -> s1 -> s2 -> s3. While rank 1 runs s1 and s2 of chunk
 *   k, rank 0 runs the exit s3 of chunk k-1 and the entry s0 of chunk k+1; with
 *   per-stage latencies tau_k growing linearly in k (Eq. 2) these two add up to
 *   the middle work (Eq. 3), so the steady state has no bubble.
 *
 *   VPP-Async (section 5.2): the same layout with rank 0's pair reordered
 *   (entry s0 of chunk k+1 before exit s3 of chunk k-1) and non-blocking
 *   transfers, so a handoff travels while the peer computes.
 *
 *   Pipelined packing (section 5.3): a rank whose next operation of the current
 *   request waits for data may run the next request's leading operations.
 *
 * Model. Operation (request r, chunk k, stage s) takes the chunk's stage time
 * (one virtual stage = a quarter of the layers; a CPP physical stage is two
 * virtual stages, so twice that). It may start when
 *   - its rank is free and it is the rank's next operation (program order, or
 *     with packing the first ready head among the requests, in request order),
 *   - (r, k, s-1) has finished, and its activation has arrived when it ran on
 *     the other rank, and
 *   - (r, k-1, s) has finished (the same layers' KV cache of the earlier chunk).
 * A handoff between ranks takes comm_time.
 *   - Synchronous mode: a handoff is a rendezvous. Both ranks reach the transfer
 *     in program order, then both are blocked for comm_time. In VPP the two
 *     handoffs of a period (chunk k+1 forward, chunk k back) form one
 *     bidirectional exchange that blocks both ranks once.
 *   - Asynchronous mode: a transfer leaves when its producer ends and arrives
 *     comm_time later; only the consumer waits.
 * Requests are queued at time 0. Without packing a rank runs requests one
 * after the other in its own program order. Ties at equal times are resolved
 * rank 0 first, then rank 1; all times are plain double sums of the inputs.
 *
 * Results: makespan, per-rank compute, exposed communication (time blocked in
 * synchronous transfers, or idle while an already finished producer's
 * activation is in flight), idle (the bubbles: the rest of the makespan), and
 * optionally every operation's interval and each request's finish time.
 */
#ifndef VPP_SCHED_H
#define VPP_SCHED_H

#include <stdint.h>

#include "vpp_chunk_attn.h" /* vpp_status_t */

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { VPP_LAYOUT_CPP = 0, VPP_LAYOUT_VPP = 1 } vpp_sched_layout_t;
typedef enum { VPP_COMM_SYNC = 0, VPP_COMM_ASYNC = 1 } vpp_sched_comm_t;

typedef struct {
    int32_t layout;            /* vpp_sched_layout_t                                  */
    int32_t comm;              /* vpp_sched_comm_t                                    */
    int32_t entry_first;       /* VPP only: rank 0 runs s0 of chunk k+1 before s3 of
                                  chunk k-1 (the reordering of section 5.2); 0 or 1  */
    int32_t packing;           /* 0 or 1; 1 requires VPP_COMM_ASYNC (section 5.3)    */
    int32_t num_requests;      /* >= 1                                                */
    const int32_t* num_chunks; /* host [num_requests], each >= 1                      */
    const double* stage_time;  /* host [sum of num_chunks]: request 0's chunks first;
                                  the time of one virtual stage of that chunk, >= 0,
                                  finite                                              */
    double comm_time;          /* one cross-rank activation handoff, >= 0, finite     */
} vpp_sched_problem_t;

typedef struct {
    double makespan;
    double compute[2];         /* per rank: sum of its operations' times            */
    double exposed_comm[2];    /* per rank: see the model above                     */
    double idle[2];            /* per rank: makespan - compute - exposed_comm       */
    double bubble_ratio;       /* (idle[0] + idle[1]) / (2 makespan); 0 if makespan 0 */
} vpp_sched_summary_t;

/* One interval of the timeline. stage is the virtual stage 0..3 (VPP) or the
 * physical stage 0..1 (CPP) of a compute operation, or -1 for a synchronous
 * transfer (then chunk is the chunk sent by that rank, or -1 for a receive
 * only). Intervals are ordered by start time, then rank. */
typedef struct {
    int32_t request, chunk, stage, rank;
    double start, end;
} vpp_sched_event_t;

/* Number of compute operations plus synchronous transfer intervals that
 * vpp_sched_simulate writes for this problem (the events capacity it needs).
 * Returns VPP_ERR_INVALID_ARG for a malformed problem. */
vpp_status_t vpp_sched_event_count(const vpp_sched_problem_t* problem, int64_t* count);

/* Run the model. summary is required. request_end (host [num_requests]) and
 * events (host [events_capacity]) are optional outputs (may be null); events
 * needs the capacity vpp_sched_event_count reports, else VPP_ERR_INVALID_ARG
 * and nothing is written. Errors: VPP_ERR_INVALID_ARG for a malformed problem
 * (null pointers, counts < 1, negative or non-finite times, packing with
 * synchronous transfers, unknown layout or mode), VPP_ERR_NOMEM when host
 * memory runs out. The call is re-entrant and owns no state. */
vpp_status_t vpp_sched_simulate(const vpp_sched_problem_t* problem, vpp_sched_summary_t* summary,
                                double* request_end, vpp_sched_event_t* events,
                                int64_t events_capacity);

#ifdef __cplusplus
}
#endif

#endif /* VPP_SCHED_H */
