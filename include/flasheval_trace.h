/*
 * flasheval_trace.h -- kernel timing of libflasheval (measurement instrumentation; it computes
 * nothing of the evaluator).
 *
 * While tracing is on, every kernel the library enqueues is bracketed by two HIP events recorded
 * on the stream the kernel is launched on, tagged with the kernel's family.  Reading the trace
 * synchronises those events and returns, per family, the summed device time and the number of
 * launches.  Tracing is process-wide and off by default; it adds two event records per launch.
 */
#ifndef FLASHEVAL_TRACE_H
#define FLASHEVAL_TRACE_H

#include <stdint.h>

#include "flasheval.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Kernel families, in the order of fe_trace_read's index. */
#define FE_TRACE_FAMILIES 12
/* 0 "gemm" (projections and the key/value cache; on fp32 models also the FFN), 1 "attention",
 * 2 "layernorm", 3 "dedup", 4 "gather", 5 "assemble", 6 "score_select", 7 "fill",
 * 8 "ffn" (kept for index stability; no kernel of this family is launched), 9 "layer" (a whole
 * encoder module -- every block and the final LayerNorm -- in one kernel, for short attention
 * groups), 10 "post" (output projection, residual, LayerNorm and FFN or query projection after
 * a separate attention kernel), 11 "linear" (the state and state-apply kernels of linear
 * attention) */

/* Turn tracing on (1) or off (0).  Turning it on discards earlier records. */
fe_status fe_trace_enable(int on);

/*
 * Synchronise every recorded event and write, for family i < FE_TRACE_FAMILIES, the summed
 * kernel time total_ms[i] and the launch count launches[i] (host arrays of FE_TRACE_FAMILIES
 * entries).  Records are consumed: a second call reports only newer launches.
 */
fe_status fe_trace_read(double* total_ms, int64_t* launches);

/*
 * Synchronise every recorded event and write the launches in the order they were enqueued:
 * family[i] and ms[i] (kernel time) for i < *count (host arrays of `capacity` entries).  If more
 * than `capacity` launches are recorded, *count receives their number, nothing else is written,
 * the records are kept and FE_EINVAL is returned.  Records are consumed otherwise.
 */
fe_status fe_trace_read_launches(int32_t* family, double* ms, int64_t capacity, int64_t* count);

/* Name of family i ("" if out of range). */
const char* fe_trace_family(int i);

#ifdef __cplusplus
}
#endif

#endif /* FLASHEVAL_TRACE_H */
