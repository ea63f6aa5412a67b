/*
 * flashkmeans.h -- C ABI of libflashkmeans.so: the exact k-means (Lloyd)
 * iteration on AMD Instinct MI355X (gfx950).
 *
 * The operations follow the Flash-KMeans workload of the paper (Section 5,
 * "Flash-KMeans clean-start workload"): a Lloyd iteration is an assignment
 * step (squared Euclidean distance of every point to every centroid, then an
 * arg-min) and a centroid update (per-cluster sums and counts of the points,
 * then their quotient).  B independent instances may be processed in one call.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All array arguments are DEVICE pointers to row-major, contiguous arrays,
 *   16-byte aligned.  The caller owns all memory; the library allocates
 *   nothing and keeps no state except a per-device architecture check.
 * - X holds B instances of N points of D dimensions: [B, N, D] in the storage
 *   type `xdtype` (FKM_F32, FKM_BF16 or FKM_F16).
 * - Centroids are fp32: [B, K, D].  The assignment rounds them once to the
 *   storage type (round-to-nearest-even) to feed the matrix cores and uses the
 *   squared norm of the rounded centroid, so each distance is the distance to
 *   that rounded centroid, accumulated in fp32.  Exception: bf16/fp16 rows of
 *   at most 16 elements run as fp32 on exactly widened copies of the points
 *   (made in the workspace), so there the distances are to the fp32
 *   centroids themselves.
 * - Indices are int32 and local to an instance: idx[b, i] is in [0, K), or -1
 *   for a point left unassigned (below).
 * - Non-finite values.  A point whose squared norm (accumulated in fp32) is
 *   not finite -- a NaN or infinite coordinate -- is left unassigned: idx -1,
 *   min_dist NaN, and it adds nothing to the objective, to any count or to
 *   any sum.  A centroid with a NaN or infinite coordinate is never chosen
 *   (it stays empty and keeps its value); a point with no other centroid is
 *   left unassigned too.  So a Lloyd run from finite centroids keeps them
 *   finite whatever NaNs the points hold.  kmeans_update skips every idx
 *   outside [0, K); the points it does sum must be finite.  Finite values
 *   whose squared norms or products overflow fp32 are outside the contract.
 *   KNN search takes finite values only.
 * - Ties go to the lowest centroid index.  An empty cluster keeps its previous
 *   centroid (and reports count 0).
 * - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and
 *   the call returns without synchronizing.  Results are deterministic:
 *   identical inputs give bit-identical outputs.
 * - A call enqueues kernel launches only (no memory set or copy commands, no
 *   host synchronization, no allocation), so it can be captured into a HIP
 *   graph and replayed; the first call on a device also reads the device's
 *   properties once, so make one call before capturing.
 * - `ws` is a device workspace of at least kmeans_workspace_bytes(...) bytes.
 *   Its contents are scratch; calls that share a workspace must be ordered on
 *   one stream.
 * - Errors: arguments are validated on the host before anything is enqueued;
 *   a rejected call returns a negative status and has no effect.
 *   FKM_ERR_UNSUPPORTED means valid but outside what this build implements:
 *   not gfx950; D > 2048; fp32 D > 256; K > 65536; N > 2^31-1; B > 65535.
 * - Row widths: the kernels take D a multiple of 16 (and, for bf16/fp16 rows
 *   wider than 256, of 32).  Any other D is served through copies of the
 *   points and centroids in zero-padded rows of the next such width, made in
 *   the workspace at the start of each call (once per kmeans_lloyd call):
 *   zeros change no distance, sum or norm, so the results are those of the
 *   unpadded rows, at the cost of that copy.  (bf16/fp16 rows of at most 16
 *   elements are copied into fp32 rows of 16, see above.)
 *   FKM_ERR_HIP reports a failed HIP call or launch.  No C++ exception
 *   crosses this boundary.
 */
#ifndef FLASHKMEANS_H_
#define FLASHKMEANS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { FKM_F32 = 0, FKM_BF16 = 1, FKM_F16 = 2 } fkm_dtype;

typedef enum {
    FKM_OK = 0,
    FKM_ERR_INVALID_ARG = -1,  /* null pointer, size < 1, bad dtype, misaligned pointer, iters < 1 */
    FKM_ERR_UNSUPPORTED = -2,  /* see the limits above */
    FKM_ERR_WORKSPACE = -3,    /* ws NULL or ws_bytes smaller than kmeans_workspace_bytes() */
    FKM_ERR_HIP = -4,          /* a HIP runtime call or a kernel launch failed */
    FKM_ERR_SCRATCH = -5       /* kmeans_lloyd_noalloc: the workspace would exceed KMEANS_SCRATCH_BYTES */
} fkm_status;

/*
 * Bytes of device workspace that kmeans_assign, kmeans_update and
 * kmeans_lloyd need for these sizes (one size serves all three).  Returns 0
 * for arguments that those calls would reject.  Pure host arithmetic.  For
 * fixed B, D, K and dtype it never decreases as N grows, so a workspace sized
 * for N serves every smaller N.
 */
size_t kmeans_workspace_bytes(int64_t B, int64_t N, int64_t D, int64_t K, int xdtype);

/*
 * Assignment step (paper Section 5: distances from each point to all K
 * centroids, then the arg-min).  The N x K distance matrix is never stored.
 *   X        [B, N, D] xdtype   points (read)
 *   C        [B, K, D] fp32     centroids (read)
 *   idx      [B, N]    int32    written: lowest k minimising ||x - c_k||^2 (-1:
 *                               unassigned, see non-finite values above)
 *   min_dist [B, N]    fp32     written: that squared distance, clamped at 0
 *                               (NaN where unassigned)
 */
int kmeans_assign(const void* X, int xdtype, const float* C, int64_t B, int64_t N, int64_t D,
                  int64_t K, int32_t* idx, float* min_dist, void* ws, size_t ws_bytes,
                  void* stream);

/*
 * Centroid update (paper Section 5: reduce the points of each cluster into a
 * per-cluster sum and count).  The reduction is a stable radix sort of the
 * point ids by cluster followed by a segmented sum in fp32 in a fixed order;
 * with few clusters (small K * D) it is per-chunk partial sums instead, added
 * in chunk order.  No floating-point atomics are used.
 *   X       [B, N, D] xdtype  points (read)
 *   idx     [B, N]    int32   cluster of each point (read); a value outside
 *                             [0, K) excludes that point from every count and sum
 *   C_prev  [B, K, D] fp32    previous centroids; rows of empty clusters are
 *                             copied to C_out (read)
 *   C_out   [B, K, D] fp32    written: sum_k / count_k (IEEE fp32 division);
 *                             may alias C_prev
 *   counts  [B, K]    int32   written: count_k
 */
int kmeans_update(const void* X, int xdtype, const int32_t* idx, const float* C_prev, int64_t B,
                  int64_t N, int64_t D, int64_t K, float* C_out, int32_t* counts, void* ws,
                  size_t ws_bytes, void* stream);

/*
 * `iters` Lloyd iterations (assignment then update), all enqueued on stream.
 *   C         [B, K, D] fp32   in: C_0, out: C_iters (updated in place)
 *   idx       [B, N]    int32  written: assignment of the last iteration
 *   min_dist  [B, N]    fp32   written: distances of the last iteration
 *   counts    [B, K]    int32  written: cluster sizes of the last iteration
 *   objective [B, iters] fp64  written if not NULL: J_t = sum_i min_dist_i of
 *                              the assignment made under C_t over the assigned
 *                              points, summed in fp64
 */
int kmeans_lloyd(const void* X, int xdtype, float* C, int64_t B, int64_t N, int64_t D, int64_t K,
                 int iters, int32_t* idx, float* min_dist, int32_t* counts, double* objective,
                 void* ws, size_t ws_bytes, void* stream);

/*
 * kmeans_lloyd for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same computation and results as kmeans_lloyd, without the `ws` argument.
 * Its workspace is a static device array of KMEANS_SCRATCH_BYTES (64 MiB)
 * inside the library, one per GPU it runs on, held until the process ends;
 * nothing is allocated by the call.  Problems whose kmeans_workspace_bytes()
 * exceeds KMEANS_SCRATCH_BYTES are rejected with FKM_ERR_SCRATCH before any
 * device work.  The caller still passes (and owns) the inputs and outputs.
 * Every call on one GPU shares that GPU's array: calls that can overlap on one
 * GPU (other streams, other host threads) race and must be serialized by the
 * caller.  The first call on a device looks the array's address up once;
 * make one call before capturing a graph.
 */
#define KMEANS_SCRATCH_BYTES ((size_t)64 << 20)
int kmeans_lloyd_noalloc(const void* X, int xdtype, float* C, int64_t B, int64_t N, int64_t D,
                         int64_t K, int iters, int32_t* idx, float* min_dist, int32_t* counts,
                         double* objective, void* stream);

/*
 * KNN search (paper Section 6 lists KNN search beside KMeans among its
 * dispatcher-backed families, with recall 1.0): for every query, the k
 * database rows at the smallest squared Euclidean distance, nearest first,
 * ties to the lowest index.  The same fused distance contraction as the
 * assignment, with a top-k in place of the arg-min; the M x N distance matrix
 * is never stored.
 *   Q        [B, M, D] xdtype   queries (read)
 *   R        [B, N, D] xdtype   database rows (read)
 *   nbr_idx  [B, M, k] int32    written: row indices, nearest first
 *   nbr_dist [B, M, k] fp32     written: their squared distances, clamped at 0
 * xdtype bf16 or fp16 (fp32 is FKM_ERR_UNSUPPORTED); D up to 256 (a D that is
 * not a multiple of 16 runs on zero-padded copies of the rows, as above);
 * 1 <= k <= min(N, 32) (k > 32 is FKM_ERR_UNSUPPORTED, k > N invalid).
 * Distances are |q|^2 - 2 <q, r> + |r|^2 with the products accumulated in fp32,
 * so rows whose distances differ by less than that rounding may trade places.
 * The workspace holds a staged copy of R (and the padded queries):
 * kmeans_knn_workspace_bytes bytes.
 */
size_t kmeans_knn_workspace_bytes(int64_t B, int64_t M, int64_t N, int64_t D, int k, int xdtype);
int kmeans_knn(const void* Q, const void* R, int xdtype, int64_t B, int64_t M, int64_t N, int64_t D,
               int k, int32_t* nbr_idx, float* nbr_dist, void* ws, size_t ws_bytes, void* stream);

/* Static, human-readable name of a status code. */
const char* kmeans_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* FLASHKMEANS_H_ */
