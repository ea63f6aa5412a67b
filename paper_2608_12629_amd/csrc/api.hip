// api.hip -- the C ABI of libflashkmeans.so (declared in include/flashkmeans.h):
// host-side argument validation, workspace carving, the gfx950 check and the
// launch sequence of each entry point.  Nothing here touches the GPU before
// the arguments have been validated.
#include <atomic>
#include <cstring>
#include <mutex>

#include "../../include/flashkmeans.h"
#include "fkm_internal.h"

namespace fkm {

static size_t align_up(size_t v) { return (v + 255) & ~size_t(255); }

// The workspace for rows of D elements; every kernel runs at w.Dk (equal to D
// unless D needs zero-padded copies of the points and centroids) in storage
// type w.kdt (the caller's, unless narrow 16-bit rows run widened to fp32).
Workspace carve(void* base, int64_t B, int64_t N, int64_t D_user, int64_t K, int dt_user) {
  Workspace w{};
  const int64_t D = kernel_dim(dt_user, D_user);
  const int dt = kernel_dt(dt_user, D_user);
  w.Dk = D;
  w.kdt = dt;
  if (assign_tiled(dt, D)) {
    w.n_assign_blocks = (N + 255) / 256;  // the decode kernel's blocks
  } else {
    const int64_t ppb = assign_points_per_block(dt, D, B * N);
    w.n_assign_blocks = (N + ppb - 1) / ppb;
  }
  // fp32 workgroups shrink to 128 points for small problems: size the
  // partials for that, so the workspace never shrinks as N grows
  const int64_t nparts = dt == DT_F32 ? (N + 127) / 128 : w.n_assign_blocks;
  w.n_sort_chunks = (N + RADIX_CHUNK - 1) / RADIX_CHUNK;
  w.red_cr = red_slice(B, N);
  w.n_red_chunks = (N + w.red_cr - 1) / w.red_cr;
  char* p = (char*)base;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    char* r = p ? p + o : nullptr;
    o = align_up(o + bytes);
    return r;
  };
  w.Kp = kpad_for(dt, D, K);
  w.chat = take((size_t)(B * w.Kp * D) * dt_bytes(dt));
  w.cinit = (float*)take((size_t)(B * w.Kp) * 4);
  w.objpart = (double*)take((size_t)(B * nparts) * 8);
  // flags of the 16-bit streaming assignment (one per block of points)
  const bool streaming16 = dt != DT_F32 && !assign_tiled(dt, D);
  w.wide = (int32_t*)take(streaming16 ? (size_t)(B * w.n_assign_blocks) * 4 : 0);
  // the second packed pass cuts at most RADIX_MAX_R more chunks (one per low digit)
  w.rhist = (int32_t*)take((size_t)(B * RADIX_MAX_R * (w.n_sort_chunks + RADIX_MAX_R)) * 4);
  w.rbin = (int32_t*)take((size_t)B * RADIX_MAX_R * 4);
  w.rbin1 = (int32_t*)take((size_t)B * RADIX_MAX_R * 4);
  w.rtotal = (int32_t*)take((size_t)B * 4);
  w.keys_a = (int32_t*)take((size_t)(B * N) * 4);
  w.vals_a = (int32_t*)take((size_t)(B * N) * 4);
  w.keys_b = (int32_t*)take((size_t)(B * N) * 4);
  w.off = (int32_t*)take((size_t)(B * (K + 1)) * 4);
  w.perm = (int32_t*)take((size_t)(B * N) * 4);
  w.carry = (float*)take((size_t)(red_slices_bound(B, N) * 2 * D) * 4);
  w.sums = (float*)take((size_t)(B * K * D) * 4);
  // per-chunk partials of the small-K update (sums_ok shapes are a subset)
  const bool sk = smallk_ok(dt, D, K);
  w.n_sk_chunks = (N + SMALLK_CH - 1) / SMALLK_CH;
  w.partial = (float*)take(sk ? (size_t)(B * w.n_sk_chunks * K * D) * 4 : 0);
  w.pcount = (int32_t*)take(sk ? (size_t)(B * w.n_sk_chunks * K) * 4 : 0);
  const bool tiled = assign_tiled(dt, D);
  w.keys = (uint64_t*)take(tiled ? (size_t)(B * N + 1) * 8 + TILED_ZERO_BYTES : 0);
  w.xnorm = (float*)take(tiled ? (size_t)(B * N) * 4 : 0);
  const bool pad = D != D_user || dt != dt_user;
  w.copied = pad;
  w.xpad = take(pad ? (size_t)(B * N * D) * dt_bytes(dt) : 0);
  w.cpad = (float*)take(pad ? (size_t)(B * K * D) * 4 : 0);
  w.total = o;
  return w;
}

// ---- validation --------------------------------------------------------------
static bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

static int check_sizes(int64_t B, int64_t N, int64_t D, int64_t K, int dt) {
  if (B < 1 || N < 1 || D < 1 || K < 1) return FKM_ERR_INVALID_ARG;
  if (dt != DT_F32 && dt != DT_BF16 && dt != DT_F16) return FKM_ERR_INVALID_ARG;
  if (N > INT32_MAX || K > MAX_K || D > MAX_D || B > 65535) return FKM_ERR_UNSUPPORTED;
  if (kernel_dim(dt, D) == 0) return FKM_ERR_UNSUPPORTED;
  return FKM_OK;
}

// Points (and centroids, when given) into the workspace's zero-padded rows
// when the kernels run at a wider row than D (and, for narrow 16-bit rows,
// widened to fp32); the pointers the kernels read.
struct KernelArgs {
  const void* X;
  float* C;
};
static hipError_t pad_inputs(const void* X, const float* C, int dt, const Workspace& w,
                             int64_t B, int64_t N, int64_t D, int64_t K, KernelArgs* a,
                             hipStream_t s) {
  a->X = X;
  a->C = const_cast<float*>(C);
  if (!w.copied) return hipSuccess;
  hipError_t e = w.kdt != dt
                     ? launch_widen_rows(X, dt, B * N, D, w.Dk, (float*)w.xpad, s)
                     : launch_pad_rows(X, B * N, D, w.Dk, dt_bytes(dt), w.xpad, s);
  if (e == hipSuccess && C) e = launch_pad_rows(C, B * K, D, w.Dk, 4, w.cpad, s);
  a->X = w.xpad;
  a->C = w.cpad;
  return e;
}

static int check_ptrs(std::initializer_list<const void*> ps) {
  for (const void* p : ps)
    if (!p || !aligned16(p)) return FKM_ERR_INVALID_ARG;
  return FKM_OK;
}

static int check_ws(void* ws, size_t ws_bytes, int64_t B, int64_t N, int64_t D, int64_t K,
                    int dt) {
  if (!ws || !aligned16(ws)) return FKM_ERR_WORKSPACE;
  if (ws_bytes < carve(nullptr, B, N, D, K, dt).total) return FKM_ERR_WORKSPACE;
  return FKM_OK;
}

// 0 = not checked yet, 1 = gfx950, 2 = other device
static std::atomic<int> g_arch[256];

static int check_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return FKM_ERR_HIP;
  if (dev < 0 || dev >= 256) return FKM_ERR_UNSUPPORTED;
  int st = g_arch[dev].load(std::memory_order_acquire);
  if (st == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return FKM_ERR_HIP;
    st = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
    if (st == 1 && update_init() != hipSuccess) return FKM_ERR_HIP;
    g_arch[dev].store(st, std::memory_order_release);
  }
  return st == 1 ? FKM_OK : FKM_ERR_UNSUPPORTED;
}

static int hip_status(hipError_t e) { return e == hipSuccess ? FKM_OK : FKM_ERR_HIP; }

// The workspace of kmeans_lloyd_noalloc: a static device array, one per GPU,
// alive until the process ends.  In host code `scratch` names a host-side
// stand-in, not device memory: its device address comes from
// hipGetSymbolAddress, once per device, and only that address is used.
static_assert(KMEANS_SCRATCH_BYTES % 256 == 0, "whole 256-byte lines");
__device__ __align__(256) char scratch[KMEANS_SCRATCH_BYTES];

static std::mutex g_scratch_mu;
static void* g_scratch_ptr[256];  // per device; nullptr until looked up

// The device address of `scratch` on the current device (looked up on the
// first call on each device).
static int scratch_on_device(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return FKM_ERR_HIP;
  if (dev < 0 || dev >= 256) return FKM_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return FKM_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return FKM_OK;
}

}  // namespace fkm

using namespace fkm;

extern "C" {

size_t kmeans_workspace_bytes(int64_t B, int64_t N, int64_t D, int64_t K, int xdtype) {
  if (check_sizes(B, N, D, K, xdtype) != FKM_OK) return 0;
  return carve(nullptr, B, N, D, K, xdtype).total;
}

int kmeans_assign(const void* X, int xdtype, const float* C, int64_t B, int64_t N, int64_t D,
                  int64_t K, int32_t* idx, float* min_dist, void* ws, size_t ws_bytes,
                  void* stream) {
  int rc;
  if ((rc = check_ptrs({X, C, idx, min_dist}))) return rc;
  if ((rc = check_sizes(B, N, D, K, xdtype))) return rc;
  if ((rc = check_ws(ws, ws_bytes, B, N, D, K, xdtype))) return rc;
  if ((rc = check_device())) return rc;
  hipStream_t s = (hipStream_t)stream;
  const Workspace w = carve(ws, B, N, D, K, xdtype);
  KernelArgs a;
  if ((rc = hip_status(pad_inputs(X, C, xdtype, w, B, N, D, K, &a, s)))) return rc;
  if ((rc = hip_status(launch_prep(a.C, w.kdt, B, K, w.Kp, w.Dk, w.chat, w.cinit, s)))) return rc;
  return hip_status(launch_assign(a.X, w.kdt, w, B, N, w.Dk, K, idx, min_dist, s));
}

int kmeans_update(const void* X, int xdtype, const int32_t* idx, const float* C_prev, int64_t B,
                  int64_t N, int64_t D, int64_t K, float* C_out, int32_t* counts, void* ws,
                  size_t ws_bytes, void* stream) {
  int rc;
  if ((rc = check_ptrs({X, idx, C_prev, C_out, counts}))) return rc;
  if ((rc = check_sizes(B, N, D, K, xdtype))) return rc;
  if ((rc = check_ws(ws, ws_bytes, B, N, D, K, xdtype))) return rc;
  if ((rc = check_device())) return rc;
  hipStream_t s = (hipStream_t)stream;
  const Workspace w = carve(ws, B, N, D, K, xdtype);
  KernelArgs a;
  if ((rc = hip_status(pad_inputs(X, C_prev, xdtype, w, B, N, D, K, &a, s)))) return rc;
  if (!w.copied)
    return hip_status(
        launch_update(X, xdtype, idx, C_prev, w, B, N, D, K, C_out, counts, NextStep{}, s));
  // copied rows: update the copy in place, then write its first D columns
  if ((rc = hip_status(
           launch_update(a.X, w.kdt, idx, a.C, w, B, N, w.Dk, K, a.C, counts, NextStep{}, s))))
    return rc;
  return hip_status(launch_unpad_rows(a.C, B * K, w.Dk, D, C_out, s));
}

int kmeans_lloyd(const void* X, int xdtype, float* C, int64_t B, int64_t N, int64_t D, int64_t K,
                 int iters, int32_t* idx, float* min_dist, int32_t* counts, double* objective,
                 void* ws, size_t ws_bytes, void* stream) {
  int rc;
  if ((rc = check_ptrs({X, C, idx, min_dist, counts}))) return rc;
  if (objective && !aligned16(objective)) return FKM_ERR_INVALID_ARG;
  if (iters < 1) return FKM_ERR_INVALID_ARG;
  if ((rc = check_sizes(B, N, D, K, xdtype))) return rc;
  if ((rc = check_ws(ws, ws_bytes, B, N, D, K, xdtype))) return rc;
  if ((rc = check_device())) return rc;
  hipStream_t s = (hipStream_t)stream;
  const Workspace w = carve(ws, B, N, D, K, xdtype);
  // padded rows are copied once; the iterations run on the copies
  KernelArgs a;
  if ((rc = hip_status(pad_inputs(X, C, xdtype, w, B, N, D, K, &a, s)))) return rc;
  const int64_t Dk = w.Dk;
  const int kdt = w.kdt;
  // Small K: one kernel assigns and sums (X read once per iteration), with
  // the arithmetic of the kernels kmeans_assign and kmeans_update run for
  // these shapes; their workgroups take SMALLK_CH points each.
  const bool fused = fused_ok(kdt, Dk, K);
  // The update's last kernel also writes the next iteration's rounded
  // centroids and scores (prep runs once) and this iteration's objective.
  NextStep nx;
  nx.dt = kdt;
  nx.chat = w.chat;
  nx.cinit = w.cinit;
  nx.Kp = w.Kp;
  nx.objpart = w.objpart;
  nx.nparts = sums_ok(kdt, Dk, K) ? w.n_sk_chunks : w.n_assign_blocks;
  nx.iters = iters;
  nx.objective = objective;
  if ((rc = hip_status(launch_prep(a.C, kdt, B, K, w.Kp, Dk, w.chat, w.cinit, s)))) return rc;
  for (int t = 0; t < iters; ++t) {
    nx.t = t;
    if (t + 1 == iters) nx.chat = nullptr;  // no next iteration
    if (fused)
      rc = hip_status(launch_sums(a.X, kdt, w, B, N, Dk, K, SUMS_FUSED, idx, min_dist, s));
    else
      rc = hip_status(launch_assign(a.X, kdt, w, B, N, Dk, K, idx, min_dist, s));
    if (rc) return rc;
    if (fused)
      rc = hip_status(launch_combine(w, w.n_sk_chunks, a.C, B, K, Dk, a.C, counts, nx, s));
    else
      rc = hip_status(launch_update(a.X, kdt, idx, a.C, w, B, N, Dk, K, a.C, counts, nx, s));
    if (rc) return rc;
  }
  if (w.copied) return hip_status(launch_unpad_rows(a.C, B * K, Dk, D, C, s));
  return FKM_OK;
}

int kmeans_lloyd_noalloc(const void* X, int xdtype, float* C, int64_t B, int64_t N, int64_t D,
                         int64_t K, int iters, int32_t* idx, float* min_dist, int32_t* counts,
                         double* objective, void* stream) {
  int rc;
  if ((rc = check_ptrs({X, C, idx, min_dist, counts}))) return rc;
  if (objective && !aligned16(objective)) return FKM_ERR_INVALID_ARG;
  if (iters < 1) return FKM_ERR_INVALID_ARG;
  if ((rc = check_sizes(B, N, D, K, xdtype))) return rc;
  if (carve(nullptr, B, N, D, K, xdtype).total > KMEANS_SCRATCH_BYTES) return FKM_ERR_SCRATCH;
  if ((rc = check_device())) return rc;
  void* ws = nullptr;
  if ((rc = scratch_on_device(&ws))) return rc;
  // the same launch sequence as kmeans_lloyd, on the static array; every
  // kernel writes its part of the workspace before reading it, so nothing
  // needs clearing between calls
  return kmeans_lloyd(X, xdtype, C, B, N, D, K, iters, idx, min_dist, counts, objective, ws,
                      KMEANS_SCRATCH_BYTES, stream);
}

// ---- KNN search ---------------------------------------------------------------
static int knn_check_sizes(int64_t B, int64_t M, int64_t N, int64_t D, int64_t k, int dt) {
  if (B < 1 || M < 1 || N < 1 || D < 1 || k < 1 || k > N) return FKM_ERR_INVALID_ARG;
  if (dt != DT_F32 && dt != DT_BF16 && dt != DT_F16) return FKM_ERR_INVALID_ARG;
  if (dt == DT_F32 || D > 256 || k > KNN_MAX_K) return FKM_ERR_UNSUPPORTED;
  if (M > INT32_MAX || N > INT32_MAX - ASSIGN_KPAD || B > 65535) return FKM_ERR_UNSUPPORTED;
  return FKM_OK;
}

// Workspace: the database rows in the staged layout [B, Np, Dk] and their
// scores [B, Np], Np = N rounded up to whole 128-row stages, Dk = D rounded up
// to a multiple of 16; when Dk != D also the queries in zero-padded rows
// [B, M, Dk].
struct KnnWs {
  void* chat;
  float* cinit;
  void* qpad;
  int64_t Np, Dk;
  size_t total;
};
static KnnWs knn_carve(void* base, int64_t B, int64_t M, int64_t N, int64_t D) {
  KnnWs w{};
  w.Np = kpad(N);
  w.Dk = (D + 15) / 16 * 16;
  char* p = (char*)base;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    char* r = p ? p + o : nullptr;
    o = align_up(o + bytes);
    return r;
  };
  w.chat = take((size_t)(B * w.Np * w.Dk) * 2);
  w.cinit = (float*)take((size_t)(B * w.Np) * 4);
  w.qpad = take(w.Dk != D ? (size_t)(B * M * w.Dk) * 2 : 0);
  w.total = o;
  return w;
}

size_t kmeans_knn_workspace_bytes(int64_t B, int64_t M, int64_t N, int64_t D, int k, int xdtype) {
  if (knn_check_sizes(B, M, N, D, k, xdtype) != FKM_OK) return 0;
  return knn_carve(nullptr, B, M, N, D).total;
}

int kmeans_knn(const void* Q, const void* R, int xdtype, int64_t B, int64_t M, int64_t N, int64_t D,
               int k, int32_t* nbr_idx, float* nbr_dist, void* ws, size_t ws_bytes, void* stream) {
  int rc;
  if ((rc = check_ptrs({Q, R, nbr_idx, nbr_dist}))) return rc;
  if ((rc = knn_check_sizes(B, M, N, D, k, xdtype))) return rc;
  if (!ws || !aligned16(ws) || ws_bytes < knn_carve(nullptr, B, M, N, D).total)
    return FKM_ERR_WORKSPACE;
  if ((rc = check_device())) return rc;
  const KnnWs w = knn_carve(ws, B, M, N, D);
  hipStream_t s = (hipStream_t)stream;
  const void* Qk = Q;
  if (w.Dk != D) {
    if ((rc = hip_status(launch_pad_rows(Q, B * M, D, w.Dk, 2, w.qpad, s)))) return rc;
    Qk = w.qpad;
  }
  if (xdtype == DT_BF16)
    return hip_status(launch_knn_bf16(Qk, R, B, M, N, D, w.Dk, k, w.chat, w.cinit, w.Np, nbr_idx,
                                      nbr_dist, s));
  return hip_status(launch_knn_f16(Qk, R, B, M, N, D, w.Dk, k, w.chat, w.cinit, w.Np, nbr_idx,
                                   nbr_dist, s));
}

const char* kmeans_status_string(int status) {
  switch (status) {
    case FKM_OK: return "ok";
    case FKM_ERR_INVALID_ARG: return "invalid argument";
    case FKM_ERR_UNSUPPORTED: return "unsupported (device or shape outside this build)";
    case FKM_ERR_WORKSPACE: return "workspace missing or too small";
    case FKM_ERR_HIP: return "HIP runtime error";
    case FKM_ERR_SCRATCH: return "problem needs more workspace than the static scratch array holds";
    default: return "unknown status";
  }
}

}  // extern "C"
