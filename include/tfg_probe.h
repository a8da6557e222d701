/*
 * Measurement probes of libtfg_probe.so: gathers with no arithmetic, used by
 * the benchmark to measure the ceiling of the row gathers that the sum
 * aggregation performs, and plain streams for the ceiling of the streaming
 * kernels (the aggregation's roofline is the rate at which the
 * CUs can pull 512-byte rows through the cache hierarchy, not HBM: the
 * gathered table of the power-law workload, 119 MB, is held by the Infinity
 * Cache). Not part of the method; the library libtfg.so does not use them.
 *
 * The two gather probes read rows of x ([rows, 128] float32, contiguous, 16-byte
 * aligned) with the aggregation's lane layout (two rows in flight per
 * wavefront instruction, 32 lanes x 16 bytes per row) and add the values into
 * registers; each wavefront writes one float of its sum to sink so that no
 * load is removed. Enqueued on `stream`; return 0, or 1 for a bad argument,
 * 6 for a launch error (the status codes of tfg.h).
 */
#ifndef TFG_PROBE_H
#define TFG_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * n_gathers rows, the i-th drawn uniformly (a fixed integer hash of i) from a
 * window of window_rows consecutive rows; the window moves to the next block
 * of window_rows rows every per_window gathers (wrapping at the end of x), as
 * the aggregation's part plan moves from one source range to the next.
 * per_window: a positive multiple of 128. sink: ceil(n_gathers / 128) floats.
 */
int tfg_probe_gather_window(const float *x, int64_t rows, int64_t window_rows,
                            int64_t n_gathers, int64_t per_window, float *sink, void *stream);

/*
 * The aggregation's own row stream without its arithmetic: item i gathers
 * the rows x[col[k]] for k in [items[2i], items[2i+1]) (at most 128 positions),
 * one wavefront per item, items in the given order (the part plan's dispatch
 * order). sink: n_items floats.
 */
int tfg_probe_gather_items(const float *x, const int32_t *col, const int32_t *items,
                           int64_t n_items, float *sink, void *stream);

/*
 * A plain stream: reads r_planes planes of n float32 words from in
 * ([r_planes, n], contiguous) and writes w_planes planes to out
 * ([max(w_planes, 1), n]), 16 bytes per thread and plane, each output word a
 * sum of the input words at its index. It measures the rate of a stream with
 * a given read / write mix (the practical ceiling of the method's streaming
 * kernels). n: a multiple of 4; in, out: 16-byte aligned. Supported mixes
 * (r_planes, w_planes): (2, 0), (1, 1), (2, 1), (2, 2), (2, 3), (8, 1);
 * any other returns 1.
 */
int tfg_probe_stream(const float *in, int r_planes, float *out, int w_planes, int64_t n,
                     void *stream);

#ifdef __cplusplus
}
#endif

#endif /* TFG_PROBE_H */
