/*
 * fkm_calib.h -- C ABI of libfkm_calib.so: microbenchmark kernels that measure,
 * on the GPU they run on and in the same process as a benchmark, the ceilings
 * against which the k-means kernels' rates are also reported (besides the
 * spec peaks): the bf16 matrix-core rate with operands that change every
 * instruction, the rate of a streaming read, and the rate of gathering whole
 * rows in a given order.  Not part of the k-means computation.
 *
 * All pointers are device pointers; each call enqueues one kernel on `stream`
 * (a hipStream_t, NULL = the null stream) and returns without synchronizing,
 * so the caller times it with events on that stream.  Returns 0, -1 for an
 * invalid argument (checked on the host before anything is enqueued), or -4
 * for a failed launch.
 */
#ifndef FKM_CALIB_H_
#define FKM_CALIB_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * bf16 matrix-core loop: `blocks` workgroups of 256 threads (2 per CU fill the
 * chip at two waves per SIMD), each wave issuing `iters` x 32 instructions of
 * 32x32x16 bf16 MFMA on 4 independent accumulators, with 8 sets of random
 * operands in rotation.  Work: blocks * 4 * iters * 32 * 32768 flops.
 *   out [blocks * 256] fp32, written (keeps the results live)
 */
int fkm_calib_mfma(float* out, int blocks, int iters, void* stream);

/*
 * Streaming read of `bytes` bytes (a multiple of 16) from `src`: each of the
 * `blocks` workgroups reads one contiguous range, 16 bytes per lane per load,
 * 8 non-temporal loads in flight.  out [blocks * 256] uint32, written.
 */
int fkm_calib_read(const void* src, size_t bytes, uint32_t* out, int blocks, void* stream);

/*
 * Gather of whole rows of `row_bytes` bytes (a multiple of 16, at most 1024)
 * from `src` (src_rows rows) in the order rows[0 .. nrows), as the segmented
 * sum reads the points: 16 bytes per lane, 8 rows in flight per lane group;
 * row indices outside [0, src_rows) are clamped into it.
 * out [blocks * 256] uint32, written.
 */
int fkm_calib_gather(const void* src, int64_t src_rows, int row_bytes, const int32_t* rows,
                     int64_t nrows, uint32_t* out, int blocks, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FKM_CALIB_H_ */
