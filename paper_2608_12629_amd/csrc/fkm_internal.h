// fkm_internal.h -- types, tuning constants and launcher declarations shared by
// the HIP translation units of libflashkmeans.so.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace fkm {

enum Dt { DT_F32 = 0, DT_BF16 = 1, DT_F16 = 2 };

__host__ __device__ inline int dt_bytes(int dt) { return dt == DT_F32 ? 4 : 2; }
constexpr int pow2_at_least(int v) { return v <= 1 ? 1 : 2 * pow2_at_least((v + 1) / 2); }

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---- tuning constants -------------------------------------------------------
// Assignment (resident-point kernels): 256 threads = 4 waves per workgroup;
// each wave keeps NSUB column tiles of points in registers; the fp32 kernel
// streams its centroids through LDS in stages of ASSIGN_TCS rows.
constexpr int ASSIGN_THREADS = 256;
constexpr int ASSIGN_TCS = 64;
// The rounded centroids and their norms are stored padded to a whole number of
// ASSIGN_KPAD-row stages: padding rows are zero with the most negative score.
constexpr int ASSIGN_KPAD = 128;
inline int64_t kpad(int64_t K) { return (K + ASSIGN_KPAD - 1) / ASSIGN_KPAD * ASSIGN_KPAD; }
// Update: the radix sort works on chunks of RADIX_CHUNK entries with digits of
// at most RADIX_MAX_BITS bits; the segmented sum gives each wave a slice of
// consecutive entries of the sorted order: the smallest power of two from
// RED_MIN to RED_MAX that keeps the slice count at or below RED_WAVES, so that
// small problems still spread over the whole chip.
constexpr int RADIX_CHUNK = 4096;
constexpr int RADIX_MAX_BITS = 8;
constexpr int RADIX_MAX_R = 1 << RADIX_MAX_BITS;
constexpr int64_t RED_MIN = 128, RED_MAX = 2048, RED_WAVES = 4096;
inline int64_t red_slice(int64_t B, int64_t N) {
  int64_t r = RED_MIN;
  while (r < RED_MAX && B * ((N + r - 1) / r) > RED_WAVES) r *= 2;
  return r;
}
// An upper bound on B * ceil(N / red_slice(B, N)) that never decreases as N
// grows, so a workspace sized for N also serves every smaller N.
inline int64_t red_slices_bound(int64_t B, int64_t N) {
  const int64_t fine = B * ((N + RED_MIN - 1) / RED_MIN);
  const int64_t coarse = B * ((N + RED_MAX - 1) / RED_MAX);
  const int64_t cap = coarse > RED_WAVES ? coarse : RED_WAVES;
  return fine < cap ? fine : cap;
}
// Small-K update: chunks of SMALLK_CH points sorted in LDS, per-chunk
// partial sums; used when K <= 512 (fp32) or 256 (16-bit), so the partials
// stay within a quarter of the rows they sum, and K * D <= SMALLK_MAX_KD.
constexpr int SMALLK_CH = 2048, SMALLK_MAX_K = 512;
constexpr int64_t SMALLK_MAX_KD = 16384;
inline bool smallk_ok(int dt, int64_t D, int64_t K) {
  return K <= (dt == DT_F32 ? 512 : 256) && K * D <= SMALLK_MAX_KD;
}
// Small-K kernels with one-hot MFMA sums (the assignment, the update's sums
// and the fused Lloyd step for these shapes): 16-bit rows of 32 to 96
// elements and at most 8 per-wave 32x32 sum tiles (128 registers): the
// ceil(K/32) cluster tiles rounded up to 2, 4 or 8, times ceil(D/32).  (Rows
// of 112 or 128 elements with their 8 tiles spill beside the three prefetched
// point tiles.)  The fused step holds the sums beside the assignment's
// registers: at most 4.
inline int64_t sums_tiles(int64_t D, int64_t K) {
  const int64_t kt = (K + 31) / 32;
  return (kt <= 2 ? 2 : (kt <= 4 ? 4 : 8)) * ((D + 31) / 32);
}
inline bool sums_ok(int dt, int64_t D, int64_t K) {
  return dt != DT_F32 && D % 16 == 0 && D >= 32 && D <= 96 && K <= 256 && sums_tiles(D, K) <= 8;
}
inline bool fused_ok(int dt, int64_t D, int64_t K) { return sums_ok(dt, D, K) && sums_tiles(D, K) <= 4; }
// KNN search: k nearest database rows per query, k <= KNN_MAX_K.
constexpr int KNN_MAX_K = 32;
// Limits of this build.
constexpr int64_t MAX_K = 65536;   // two radix passes of at most 8 bits
constexpr int64_t MAX_D = 2048;

// Row widths the kernels handle: D a multiple of 16 (rows of whole 32-byte
// or 64-byte pieces), at most 8 KiB per row.
inline bool row_bytes_ok(int dt, int64_t D) {
  return D % 16 == 0 && D >= 16 && D * dt_bytes(dt) <= 8192;
}

// Points per assignment workgroup.  16-bit storage: 32x32x16 MFMA tiles, 4
// waves x NSUB x 32 points, NSUB by the D / 16 chunks a lane holds (4 up to 4
// chunks, 2 up to 8, else 1).  fp32: 16x16x4 MFMA tiles, 4 waves x NSUB x 16
// points (NSUB = 8 up to D = 64, 4 up to 128, else 2), and 2 when B x N
// points would give fewer than 512 workgroups (two per CU) at the larger
// NSUB: a small problem then fills the chip with smaller workgroups.
inline int assign_nsub16(int64_t D) { return D <= 64 ? 4 : (D <= 128 ? 2 : 1); }
inline int assign_nsub32(int64_t D, int64_t BN) {
  const int base = D <= 64 ? 8 : (D <= 128 ? 4 : 2);
  return base > 2 && BN < (int64_t)512 * 64 * base ? 2 : base;
}
inline int64_t assign_points_per_block(int dt, int64_t D, int64_t BN) {
  if (dt != DT_F32) return 4 * 32 * assign_nsub16(D);
  return 4 * 16 * assign_nsub32(D, BN);
}

// The resident-X assignment kernels hold a point in registers: rows up to
// D = 256.  Wider 16-bit rows with D a multiple of 32 go to the tiled kernel.
inline bool assign_resident_ok(int dt, int64_t D) { return D % 16 == 0 && D >= 16 && D <= 256; }
inline bool assign_tiled(int dt, int64_t D) { return dt != DT_F32 && D > 256 && D % 32 == 0; }
inline bool assign_ok(int dt, int64_t D) { return assign_resident_ok(dt, D) || assign_tiled(dt, D); }
// The row width the kernels run at: D itself when they take it, else D
// rounded up to a multiple of 16 (32 for 16-bit rows wider than 256), with the
// points and centroids copied into zero-padded rows first (zeros change no
// distance, sum or norm).  0 when no kernel takes the rounded width either.
inline int64_t kernel_dim(int dt, int64_t D) {
  if (D < 1 || D > MAX_D) return 0;
  if (row_bytes_ok(dt, D) && assign_ok(dt, D)) return D;
  const int64_t Dk = D <= 256 ? (D + 15) / 16 * 16 : (D + 31) / 32 * 32;
  return row_bytes_ok(dt, Dk) && assign_ok(dt, Dk) ? Dk : 0;
}
// The storage type the kernels run in: the caller's, except for 16-bit rows
// of at most 16 elements, which run as fp32 on widened (exact) copies.
// Their centroids then enter the distances unrounded: rounding a centroid to
// the 16-bit type moves a distance by about 2 <x - c, c - c^>, at most
// 2 |x - c| 2^-9 |c| for bf16, which averages out over many dimensions but
// over a handful is not small against 1e-3 |x|^2 when a point's nearest
// centroids are far from it relative to its norm.
inline int kernel_dt(int dt, int64_t D) { return dt != DT_F32 && D <= 16 ? DT_F32 : dt; }
// Tiled kernel: 256 points x 256-centroid blocks, TILED_CBG blocks per
// workgroup; its centroids are padded to whole blocks.
constexpr int TILED_BP = 256, TILED_BC = 256, TILED_CBG = 8;
constexpr int64_t TILED_ZERO_BYTES = 16384;  // zeros after the keys (padding stages)
inline int64_t kpad_for(int dt, int64_t D, int64_t K) {
  return assign_tiled(dt, D) ? (K + TILED_BC - 1) / TILED_BC * TILED_BC : kpad(K);
}

// ---- workspace layout -------------------------------------------------------
struct Workspace {
  void* chat;      // [B,Kp,D] centroids rounded to the storage type (Kp = kpad_for(dt, D, K))
  float* cinit;    // [B,Kp]   -1/2 * squared norm of each rounded centroid
  double* objpart; // [B,n_assign_blocks] per-workgroup objective partials
  int32_t* wide;   // [B,n_assign_blocks] blocks whose norms spread widely (16-bit streaming assignment)
  int32_t* rhist;  // [B,R,chunks] radix histograms, then run starts (R <= 256; chunks <= n_sort_chunks + 256)
  int32_t* rbin;   // [B,256] radix bin totals
  int32_t* rbin1;  // [B,256] the first pass's bin totals (packed two-pass sort)
  int32_t* rtotal; // [B] number of valid entries (ids in [0, K))
  int32_t* keys_a; // [B,N] cluster ids after the first radix pass
  int32_t* vals_a; // [B,N] point ids after the first radix pass
  int32_t* keys_b; // [B,N] cluster ids, sorted
  int32_t* off;    // [B,K+1] cluster start offsets in the sorted order
  int32_t* perm;   // [B,N] point ids sorted by cluster
  float* carry;    // [B,n_red_chunks,2,D] partial sums of clusters cut by slice ends
  float* sums;     // [B,K,D] sums of clusters that fit in one chunk
  float* partial;  // [B,nch,K,D] per-chunk cluster sums (small-K update; nch = n_sk_chunks, or n_assign_blocks when sums_ok)
  int32_t* pcount; // [B,nch,K] per-chunk cluster counts
  uint64_t* keys;  // [B,N] best (score, index) of each point, then TILED_ZERO_BYTES of zeros (tiled assignment only)
  float* xnorm;    // [B,N] squared norms of the points (tiled assignment only)
  void* xpad;      // [B,N,Dk] the points in zero-padded rows of type kdt (only when copied)
  float* cpad;     // [B,K,Dk] the centroids in zero-padded rows (only when copied)
  int64_t Dk;      // the row width the kernels run at (kernel_dim)
  int kdt;         // the storage type the kernels run in (kernel_dt)
  bool copied;     // the kernels read copies (xpad, cpad): Dk != D or kdt != the caller's type
  int64_t Kp, n_assign_blocks, n_sort_chunks, n_red_chunks, red_cr, n_sk_chunks;
  size_t total;
};

Workspace carve(void* base, int64_t B, int64_t N, int64_t D, int64_t K, int dt);

// What the update's last kernel also produces inside kmeans_lloyd: the next
// iteration's assignment inputs (the rounded centroids and their scores, as
// prep would write them) and the objective of this iteration's assignment.
struct NextStep {
  int dt = 0;
  void* chat = nullptr;          // [B,Kp,D]; nullptr: not written
  float* cinit = nullptr;        // [B,Kp]
  int64_t Kp = 0;
  const double* objpart = nullptr;
  int64_t nparts = 0;            // objective partials per instance
  int iters = 0, t = 0;
  double* objective = nullptr;   // [B,iters]; nullptr: not computed
};

// ---- launchers (return hipSuccess or the launch error) ----------------------
hipError_t launch_prep(const float* C, int dt, int64_t B, int64_t K, int64_t Kp, int64_t D,
                       void* chat, float* cinit, hipStream_t s);
hipError_t launch_assign(const void* X, int dt, const Workspace& w, int64_t B, int64_t N,
                         int64_t D, int64_t K, int32_t* idx, float* min_dist, hipStream_t s);
hipError_t launch_pipe_bf16(const void* X, const Workspace& w, int64_t B, int64_t N, int64_t D,
                           int32_t* idx, float* min_dist, hipStream_t s);
hipError_t launch_pipe_f16(const void* X, const Workspace& w, int64_t B, int64_t N, int64_t D,
                          int32_t* idx, float* min_dist, hipStream_t s);
// sums_ok shapes, by mode: SUMS_ASSIGN the assignment (idx, min_dist and
// objective partials, one per SMALLK_CH points), SUMS_FUSED that plus the
// per-chunk partial sums and counts, SUMS_ONLY the partials of the given idx.
enum SumsMode { SUMS_ASSIGN = 0, SUMS_FUSED = 1, SUMS_ONLY = 2 };
hipError_t launch_sums_bf16(const void* X, const Workspace& w, int64_t B, int64_t N, int64_t D,
                           int64_t K, int mode, int32_t* idx, float* min_dist, hipStream_t s);
hipError_t launch_sums_f16(const void* X, const Workspace& w, int64_t B, int64_t N, int64_t D,
                          int64_t K, int mode, int32_t* idx, float* min_dist, hipStream_t s);
hipError_t launch_sums(const void* X, int dt, const Workspace& w, int64_t B, int64_t N, int64_t D,
                       int64_t K, int mode, int32_t* idx, float* min_dist, hipStream_t s);
// Means from the per-chunk partials and counts (nch chunks per instance).
hipError_t launch_combine(const Workspace& w, int64_t nch, const float* C_prev, int64_t B,
                          int64_t K, int64_t D, float* C_out, int32_t* counts,
                          const NextStep& nx, hipStream_t s);
// KNN: R rows of Din elements; Q rows and the staged rows of D >= Din (a multiple of 16)
hipError_t launch_knn_bf16(const void* Q, const void* R, int64_t B, int64_t M, int64_t N,
                           int64_t Din, int64_t D, int k, void* chat, float* cinit, int64_t Np,
                           int32_t* nbr_idx, float* nbr_dist, hipStream_t s);
hipError_t launch_knn_f16(const void* Q, const void* R, int64_t B, int64_t M, int64_t N,
                          int64_t Din, int64_t D, int k, void* chat, float* cinit, int64_t Np,
                          int32_t* nbr_idx, float* nbr_dist, hipStream_t s);
hipError_t launch_assign_tiled(const void* X, int dt, const Workspace& w, int64_t B, int64_t N,
                               int64_t D, int32_t* idx, float* min_dist, hipStream_t s);
hipError_t launch_pad_rows(const void* src, int64_t rows, int64_t D, int64_t Dk, int elem_bytes,
                           void* dst, hipStream_t s);
// 16-bit rows of D elements (dt) into fp32 rows of Dk >= D (zeros past D).
hipError_t launch_widen_rows(const void* src, int dt, int64_t rows, int64_t D, int64_t Dk,
                             float* dst, hipStream_t s);
hipError_t launch_unpad_rows(const float* src, int64_t rows, int64_t Dk, int64_t D, float* dst,
                             hipStream_t s);
hipError_t update_init();
hipError_t launch_update(const void* X, int dt, const int32_t* idx, const float* C_prev,
                         const Workspace& w, int64_t B, int64_t N, int64_t D, int64_t K,
                         float* C_out, int32_t* counts, const NextStep& nx, hipStream_t s);

}  // namespace fkm
