/*
 * m2r2_measure.h -- measurement hooks of libm2r2.so, outside the decode
 * path's boundary (include/m2r2.h).  They time kernel classes of the decode
 * pass with HIP events so that a benchmark can report one kernel's duration
 * against its algorithmic bytes; no decode result depends on them.
 */
#ifndef M2R2_MEASURE_H_
#define M2R2_MEASURE_H_

#include "m2r2.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Kernel timing for measurement.  Kernel classes of one decode pass:
 * 0 qkv, 1 attention, 2 output projection, 3 gate/up, 4 down, 5 LM head,
 * 6 embedding, 7 attention merge, 8 expert gate/up, 9 expert down, 10
 * router and top-k, 11 the one-launch decode step of one sequence (every
 * layer and the head in one kernel).  m2r2_timing_enable(ctx, k) starts a new record: every
 * launch of class k made by later calls is bracketed by a pair of HIP events
 * recorded on the call's stream (up to 1024 launches; record with direct
 * launches: events recorded inside a captured graph cannot be timed).
 * m2r2_timing_read waits for the recorded events and returns the summed
 * kernel milliseconds and the launch count of the record.  k = -1 stops
 * recording.  Events are host-side objects created by the library (no device
 * memory). */
M2R2_API m2r2_status m2r2_timing_enable(m2r2_ctx* ctx, int32_t kernel_class);
M2R2_API m2r2_status m2r2_timing_read(m2r2_ctx* ctx, double* ms_sum, int32_t* launches);

/* Average duration of one gate/up launch (kernel class 3) of the
 * one-sequence decode step (two rows when `dual`, one otherwise): the kernel
 * of every layer is launched back to back on `stream` between one pair of HIP
 * events (which keeps the events' own latency out of the per-launch figure;
 * each layer streams its own weights, as in a step), and *avg_ms receives the
 * elapsed time divided by the layer count.  Waits for `stream`.  Side
 * effects: the workspace's SwiGLU activations and the gate/up row statistics
 * (zeroed at the start of every pass) are overwritten; the residual stream,
 * the cache and the positions are not touched.  Returns M2R2_E_UNSUPPORTED
 * when the one- and two-row decode class does not use the row-per-wave
 * kernels (for example a mixture-of-experts model). */
M2R2_API m2r2_status m2r2_time_gateup_layers(m2r2_ctx* ctx, int32_t dual, hipStream_t stream, double* avg_ms);

#ifdef __cplusplus
}
#endif
#endif /* M2R2_MEASURE_H_ */
