// extern "C" boundary of libnystra: argument validation, option resolution,
// kernel-family selection and launch.  Every check runs before anything is
// enqueued; the layer allocates nothing and never synchronises.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <mutex>

#include "../../include/nystra.h"
#include "internal.hpp"

namespace nystra {

bool make_geometry(int N, int m, int mode, Geometry *g)
{
    if (N < 1 || m < 1 || m > N)
        return false;
    if (mode == NYSTRA_LM_POOL2D) {
        int w = int(sqrt(double(N)) + 0.5);
        if (w * w != N)
            return false;
        int best = 0;
        for (int gc = 1; gc * gc <= m; ++gc)
            if (m % gc == 0 && w % gc == 0 && w % (m / gc) == 0)
                best = gc;
        if (best == 0)
            return false;
        *g = Geometry{w, w, w / (m / best), w / best, best};
        return true;
    }
    if (mode == NYSTRA_LM_SEGMENT1D) {
        if (N % m != 0)
            return false;
        *g = Geometry{1, N, 1, N / m, m};
        return true;
    }
    return false;
}

size_t generic_lds_bytes(int m, int d);

}  // namespace nystra

using nystra::Problem;

namespace {

// Tokens per window: up to 2^20 (a 1024 x 1024 map as one global window).  The
// kernels stream over tokens with 64-bit offsets and size LDS independently of N.
constexpr int kMaxN = 1 << 20;
constexpr int kMaxD = 128;
constexpr int kMaxM = 64;
constexpr int kMaxIters = 64;
// Units per call: every kernel's grid is at most 256 work-items per unit in its
// x dimension, and a launch holds fewer than 2^32 work-items per dimension.
constexpr int64_t kMaxUnits = (int64_t(1) << 24) - 1;

thread_local char g_last_error[256] = "";

void set_last_error(const char *msg)
{
    strncpy(g_last_error, msg ? msg : "", sizeof(g_last_error) - 1);
    g_last_error[sizeof(g_last_error) - 1] = '\0';
}

int dtype_bytes(int dtype) { return dtype == NYSTRA_F32 ? 4 : 2; }

bool misaligned(const void *p, int bytes) { return (uintptr_t(p) % uintptr_t(bytes)) != 0; }

bool overlaps(const void *a, int64_t an, const void *b, int64_t bn)
{
    const uintptr_t a0 = uintptr_t(a), b0 = uintptr_t(b);
    return a0 < b0 + uintptr_t(bn) && b0 < a0 + uintptr_t(an);
}

// Shape, dtype and count checks shared by every device entry point.
int check_common(int n_windows, int heads, int N, int d, int dtype, int64_t *units)
{
    if (dtype != NYSTRA_F32 && dtype != NYSTRA_BF16)
        return NYSTRA_ERR_DTYPE;
    if (n_windows < 0 || heads < 0 || N < 1 || N > kMaxN || d < 1 || d > kMaxD)
        return NYSTRA_ERR_SHAPE;
    const int64_t u = int64_t(n_windows) * int64_t(heads);
    if (u > kMaxUnits)
        return NYSTRA_ERR_SHAPE;
    *units = u;
    return NYSTRA_OK;
}

// Pointer checks: non-null, element-aligned, O disjoint from the inputs.
int check_tensors(const void *Q, const void *K, const void *V, const void *O, int64_t bytes,
                  int ebytes)
{
    if (!Q || !K || !V || !O)
        return NYSTRA_ERR_NULL;
    if (misaligned(Q, ebytes) || misaligned(K, ebytes) || misaligned(V, ebytes) ||
        misaligned(O, ebytes))
        return NYSTRA_ERR_ALIGN;
    if (overlaps(O, bytes, Q, bytes) || overlaps(O, bytes, K, bytes) ||
        overlaps(O, bytes, V, bytes))
        return NYSTRA_ERR_OVERLAP;
    return NYSTRA_OK;
}

// hipGetLastError() reports the last error of any HIP call on this thread.
// Each entry point clears it right before its first launch, so that the
// status it returns speaks of its own launches only.
void clear_stale_error() { (void)hipGetLastError(); }

int finish_launch(hipError_t e)
{
    if (e != hipSuccess) {
        set_last_error(hipGetErrorString(e));
        return NYSTRA_ERR_HIP;
    }
    return NYSTRA_OK;
}

// Token-split kernels pay off for long windows: from 64 x 64 tokens on they beat
// one workgroup per unit at every unit count measured (384 to 1536 units),
// from 2048 tokens when the units are too few to fill the GPU (< 512).  At
// 32 x 32 windows with 1536 units the one-pass kernel is faster.
bool split_preferred(const Problem &p)
{
    return p.N >= 4096 || (p.N >= 2048 && p.units < 512);
}

// Resolves options and the problem; does not touch device memory.  with_ws
// says whether the entry point takes a workspace (and so may run the
// token-split kernels).
int build_problem(const void *Q, const void *K, const void *V, void *O, int n_windows,
                  int heads, int N, int d, int m, int dtype, const nystra_opts *opts,
                  bool with_ws, Problem *p, int *variant)
{
    nystra_opts o;
    nystra_default_opts(&o);
    if (opts)
        o = *opts;
    int64_t units = 0;
    int rc = check_common(n_windows, heads, N, d, dtype, &units);
    if (rc != NYSTRA_OK)
        return rc;
    if (m < 1 || m > N || m > kMaxM)
        return NYSTRA_ERR_SHAPE;
    if (o.pinv_iters < 0 || o.pinv_iters > kMaxIters || !isfinite(o.scale) ||
        (o.landmark_mode != NYSTRA_LM_POOL2D && o.landmark_mode != NYSTRA_LM_SEGMENT1D) ||
        o.variant < NYSTRA_VARIANT_AUTO || o.variant > NYSTRA_VARIANT_SPLIT)
        return NYSTRA_ERR_ARG;
    nystra::Geometry g;
    if (!nystra::make_geometry(N, m, o.landmark_mode, &g))
        return NYSTRA_ERR_SHAPE;
    p->q = Q;
    p->k = K;
    p->v = V;
    p->o = O;
    p->units = units;
    p->N = N;
    p->d = d;
    p->m = m;
    p->iters = o.pinv_iters;
    p->dtype = dtype;
    p->scale = o.scale > 0.f ? o.scale : float(1.0 / sqrt(double(d)));
    p->geo = g;
    const bool tiled = nystra::tiled_supported(*p);
    const bool split = with_ws && nystra::split_supported(*p);
    switch (o.variant) {
    case NYSTRA_VARIANT_GENERIC:
        *variant = NYSTRA_VARIANT_GENERIC;
        return NYSTRA_OK;
    case NYSTRA_VARIANT_TILED:
        *variant = NYSTRA_VARIANT_TILED;
        return tiled ? NYSTRA_OK : NYSTRA_ERR_UNSUPPORTED;
    case NYSTRA_VARIANT_SPLIT:
        *variant = NYSTRA_VARIANT_SPLIT;
        return split ? NYSTRA_OK : NYSTRA_ERR_UNSUPPORTED;
    default:
        *variant = (split && split_preferred(*p)) ? NYSTRA_VARIANT_SPLIT
                   : tiled                        ? NYSTRA_VARIANT_TILED
                                                  : NYSTRA_VARIANT_GENERIC;
        return NYSTRA_OK;
    }
}

}  // namespace

extern "C" {

int nystra_default_opts(nystra_opts *opts)
{
    if (!opts)
        return NYSTRA_ERR_NULL;
    opts->pinv_iters = 6;
    opts->landmark_mode = NYSTRA_LM_POOL2D;
    opts->scale = 0.f;
    opts->variant = NYSTRA_VARIANT_AUTO;
    return NYSTRA_OK;
}

int nystra_attn_forward_ex(const void *Q, const void *K, const void *V, void *O, int n_windows,
                           int heads, int N, int d_h, int m, int dtype, const nystra_opts *opts,
                           void *stream)
{
    Problem p;
    int variant = 0;
    int rc = build_problem(Q, K, V, O, n_windows, heads, N, d_h, m, dtype, opts, false, &p,
                           &variant);
    if (rc != NYSTRA_OK)
        return rc;
    if (p.units == 0)
        return NYSTRA_OK;
    const int64_t bytes = p.units * N * d_h * dtype_bytes(dtype);
    rc = check_tensors(Q, K, V, O, bytes, dtype_bytes(dtype));
    if (rc != NYSTRA_OK)
        return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    clear_stale_error();
    if (variant == NYSTRA_VARIANT_TILED)
        return finish_launch(nystra::launch_tiled_forward(p, s));
    return finish_launch(nystra::launch_generic_forward(p, s));
}

int nystra_attn_workspace_size(int n_windows, int heads, int N, int d_h, int m, int dtype,
                               const nystra_opts *opts, size_t *bytes)
{
    if (!bytes)
        return NYSTRA_ERR_NULL;
    Problem p;
    int variant = 0;
    int rc = build_problem(nullptr, nullptr, nullptr, nullptr, n_windows, heads, N, d_h, m,
                           dtype, opts, true, &p, &variant);
    if (rc != NYSTRA_OK)
        return rc;
    *bytes = (variant == NYSTRA_VARIANT_SPLIT && p.units > 0)
                 ? nystra::split_workspace_bytes(p) : 0;
    return NYSTRA_OK;
}

int nystra_attn_forward_ws(const void *Q, const void *K, const void *V, void *O,
                           int n_windows, int heads, int N, int d_h, int m, int dtype,
                           const nystra_opts *opts, void *workspace, size_t workspace_bytes,
                           void *stream)
{
    Problem p;
    int variant = 0;
    int rc = build_problem(Q, K, V, O, n_windows, heads, N, d_h, m, dtype, opts, true, &p,
                           &variant);
    if (rc != NYSTRA_OK)
        return rc;
    if (p.units == 0)
        return NYSTRA_OK;
    const int64_t bytes = p.units * N * d_h * dtype_bytes(dtype);
    rc = check_tensors(Q, K, V, O, bytes, dtype_bytes(dtype));
    if (rc != NYSTRA_OK)
        return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (variant == NYSTRA_VARIANT_SPLIT) {
        const size_t need = nystra::split_workspace_bytes(p);
        if (!workspace || workspace_bytes < need || misaligned(workspace, 256))
            return NYSTRA_ERR_WORKSPACE;
        const int64_t wn = int64_t(need);
        if (overlaps(workspace, wn, Q, bytes) || overlaps(workspace, wn, K, bytes) ||
            overlaps(workspace, wn, V, bytes) || overlaps(workspace, wn, O, bytes))
            return NYSTRA_ERR_WORKSPACE;
        clear_stale_error();
        return finish_launch(nystra::launch_split(p, workspace, s));
    }
    clear_stale_error();
    if (variant == NYSTRA_VARIANT_TILED)
        return finish_launch(nystra::launch_tiled_forward(p, s));
    return finish_launch(nystra::launch_generic_forward(p, s));
}

}  // extern "C"

namespace {

// Scratch of the allocation-free entry point: the token-split workspace as a
// static device array.  Every device the library runs on holds its own copy
// at its own address, until the process ends.  In host code `scratch` names a
// host-side stand-in only; kernels receive the device address looked up below.
static __device__ __align__(256) unsigned char scratch[NYSTRA_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on device `dev`, looked up once per device with
// that device current (the caller's current device, checked by the caller).
hipError_t scratch_address(int dev, void **ptr)
{
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

extern "C" {

int nystra_attn_forward_noalloc(const void *Q, const void *K, const void *V, void *O,
                                int n_windows, int heads, int N, int d_h, int m, int dtype,
                                const nystra_opts *opts, void *stream)
{
    Problem p;
    int variant = 0;
    int rc = build_problem(Q, K, V, O, n_windows, heads, N, d_h, m, dtype, opts, true, &p,
                           &variant);
    if (rc != NYSTRA_OK)
        return rc;
    if (p.units == 0)
        return NYSTRA_OK;
    const int64_t bytes = p.units * N * d_h * dtype_bytes(dtype);
    rc = check_tensors(Q, K, V, O, bytes, dtype_bytes(dtype));
    if (rc != NYSTRA_OK)
        return rc;
    const size_t need = variant == NYSTRA_VARIANT_SPLIT ? nystra::split_workspace_bytes(p) : 0;
    if (need > size_t(NYSTRA_STATIC_SCRATCH_BYTES)) {
        set_last_error("token-split workspace exceeds NYSTRA_STATIC_SCRATCH_BYTES");
        return NYSTRA_ERR_WORKSPACE;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    clear_stale_error();
    if (variant != NYSTRA_VARIANT_SPLIT) {   // these kernels use no scratch memory
        if (variant == NYSTRA_VARIANT_TILED)
            return finish_launch(nystra::launch_tiled_forward(p, s));
        return finish_launch(nystra::launch_generic_forward(p, s));
    }
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return finish_launch(e);
    if (dev < 0 || dev >= kMaxDevices) {
        set_last_error("device index beyond the scratch table");
        return NYSTRA_ERR_ARG;
    }
    if (s) {   // the kernels run on the stream's device; its scratch copy must be the one used
        int sdev = -1;
        e = hipStreamGetDevice(s, &sdev);
        if (e != hipSuccess)
            return finish_launch(e);
        if (sdev != dev) {
            set_last_error("stream does not belong to the current device");
            return NYSTRA_ERR_ARG;
        }
    }
    void *ws = nullptr;
    e = scratch_address(dev, &ws);
    if (e != hipSuccess)
        return finish_launch(e);
    return finish_launch(nystra::launch_split(p, ws, s));
}

int nystra_attn_forward(const void *Q, const void *K, const void *V, void *O, int n_windows,
                        int heads, int N, int d_h, int m, int dtype, void *stream)
{
    return nystra_attn_forward_ex(Q, K, V, O, n_windows, heads, N, d_h, m, dtype, nullptr,
                                  stream);
}

int nystra_exact_attn_forward(const void *Q, const void *K, const void *V, void *O,
                              int n_windows, int heads, int N, int d_h, int dtype, float scale,
                              void *stream)
{
    int64_t units = 0;
    int rc = check_common(n_windows, heads, N, d_h, dtype, &units);
    if (rc != NYSTRA_OK)
        return rc;
    if (!isfinite(scale))
        return NYSTRA_ERR_ARG;
    if (units == 0)
        return NYSTRA_OK;
    const int64_t bytes = units * N * d_h * dtype_bytes(dtype);
    rc = check_tensors(Q, K, V, O, bytes, dtype_bytes(dtype));
    if (rc != NYSTRA_OK)
        return rc;
    Problem p{};
    p.q = Q;
    p.k = K;
    p.v = V;
    p.o = O;
    p.units = units;
    p.N = N;
    p.d = d_h;
    p.m = 0;
    p.dtype = dtype;
    p.scale = scale > 0.f ? scale : float(1.0 / sqrt(double(d_h)));
    clear_stale_error();
    return finish_launch(nystra::launch_exact(p, static_cast<hipStream_t>(stream)));
}

int nystra_landmark_pool(const void *Q, const void *K, float *Qbar, float *Kbar, int32_t *map,
                         int n_windows, int heads, int N, int d_h, int m, int dtype, int mode,
                         void *stream)
{
    int64_t units = 0;
    int rc = check_common(n_windows, heads, N, d_h, dtype, &units);
    if (rc != NYSTRA_OK)
        return rc;
    if (m < 1 || m > N || m > kMaxM)
        return NYSTRA_ERR_SHAPE;
    if (mode != NYSTRA_LM_POOL2D && mode != NYSTRA_LM_SEGMENT1D)
        return NYSTRA_ERR_ARG;
    nystra::Geometry g;
    if (!nystra::make_geometry(N, m, mode, &g))
        return NYSTRA_ERR_SHAPE;
    if (units == 0)
        return NYSTRA_OK;
    const int eb = dtype_bytes(dtype);
    if (!Q || !K || !Qbar || !Kbar)
        return NYSTRA_ERR_NULL;
    if (misaligned(Q, eb) || misaligned(K, eb) || misaligned(Qbar, 4) || misaligned(Kbar, 4) ||
        (map && misaligned(map, 4)))
        return NYSTRA_ERR_ALIGN;
    const int64_t in_bytes = units * N * d_h * eb, out_bytes = units * m * d_h * 4;
    if (overlaps(Qbar, out_bytes, Q, in_bytes) || overlaps(Qbar, out_bytes, K, in_bytes) ||
        overlaps(Kbar, out_bytes, Q, in_bytes) || overlaps(Kbar, out_bytes, K, in_bytes) ||
        overlaps(Qbar, out_bytes, Kbar, out_bytes))
        return NYSTRA_ERR_OVERLAP;
    Problem p{};
    p.q = Q;
    p.k = K;
    p.units = units;
    p.N = N;
    p.d = d_h;
    p.m = m;
    p.dtype = dtype;
    p.geo = g;
    clear_stale_error();
    return finish_launch(
        nystra::launch_landmark_pool(p, Qbar, Kbar, map, static_cast<hipStream_t>(stream)));
}

int nystra_landmark_map(int N, int m, int mode, int32_t *map_host)
{
    if (mode != NYSTRA_LM_POOL2D && mode != NYSTRA_LM_SEGMENT1D)
        return NYSTRA_ERR_ARG;
    if (N < 1 || N > kMaxN || m < 1 || m > N || m > kMaxM)
        return NYSTRA_ERR_SHAPE;
    nystra::Geometry g;
    if (!nystra::make_geometry(N, m, mode, &g))
        return NYSTRA_ERR_SHAPE;
    if (!map_host)
        return NYSTRA_ERR_NULL;
    for (int t = 0; t < N; ++t) {
        const int r = t / g.cols, c = t % g.cols;
        map_host[t] = (r / g.pr) * g.gc + c / g.pc;
    }
    return NYSTRA_OK;
}

int nystra_select_variant(int N, int d_h, int m, int dtype, const nystra_opts *opts)
{
    Problem p;
    int variant = 0;
    int rc = build_problem(nullptr, nullptr, nullptr, nullptr, 1, 1, N, d_h, m, dtype, opts,
                           false, &p, &variant);
    return rc == NYSTRA_OK ? variant : -rc;
}

}  // extern "C"

namespace {

// Workspace layout of the block: Q, K, V, O, the packed weights of the two
// GEMMs (when C <= 256), then the attention's own.
struct BlockPlan {
    Problem p;          // the attention problem on the workspace tensors
    int variant;        // attention kernel family (Nystrom) or -1 (exact)
    size_t qkvo_bytes;  // one of the four tensors, padded to 256 bytes
    size_t pk_qkv, pk_proj;   // packed W_qkv and W_proj, padded to 256 bytes (0: none)
    size_t bytes;       // total
};

size_t pad256(size_t x) { return (x + 255) & ~size_t(255); }

int plan_block(const nystra_block_shape *s, int m, int dtype, const nystra_opts *opts,
               int attention, BlockPlan *bp)
{
    if (!s)
        return NYSTRA_ERR_NULL;
    if (dtype != NYSTRA_F32 && dtype != NYSTRA_BF16)
        return NYSTRA_ERR_DTYPE;
    if (attention != NYSTRA_BLOCK_NYSTROM && attention != NYSTRA_BLOCK_EXACT)
        return NYSTRA_ERR_ARG;
    if (s->batch < 0 || s->height < 1 || s->width < 1 || s->window < 1 || s->heads < 1 ||
        s->channels < 1 || s->channels > 4096 || s->channels % s->heads != 0 ||
        s->height % s->window != 0 || s->width % s->window != 0 || s->shift < 0 ||
        s->shift >= s->window || s->window > 1024)
        return NYSTRA_ERR_SHAPE;
    const int64_t rows = int64_t(s->batch) * s->height * s->width;
    if (rows > int64_t(INT32_MAX) || !nystra::block_gemm_supported(rows, s->channels))
        return NYSTRA_ERR_SHAPE;
    const int64_t nw = int64_t(s->batch) * (s->height / s->window) * (s->width / s->window);
    if (nw > int64_t(INT32_MAX))
        return NYSTRA_ERR_SHAPE;
    const int N = s->window * s->window, d = s->channels / s->heads;
    int rc;
    if (attention == NYSTRA_BLOCK_NYSTROM) {
        rc = build_problem(nullptr, nullptr, nullptr, nullptr, int(nw), s->heads, N, d, m, dtype,
                           opts, true, &bp->p, &bp->variant);
    } else {
        int64_t units = 0;
        rc = check_common(int(nw), s->heads, N, d, dtype, &units);
        if (rc == NYSTRA_OK && opts && !isfinite(opts->scale))
            rc = NYSTRA_ERR_ARG;
        bp->p = Problem{};
        bp->p.units = units;
        bp->p.N = N;
        bp->p.d = d;
        bp->p.dtype = dtype;
        const float sc = opts ? opts->scale : 0.f;
        bp->p.scale = sc > 0.f ? sc : float(1.0 / sqrt(double(d)));
        bp->variant = -1;
    }
    if (rc != NYSTRA_OK)
        return rc;
    bp->qkvo_bytes = pad256(size_t(rows) * s->channels * dtype_bytes(dtype));
    bp->pk_qkv = pad256(nystra::block_wpack_bytes(s->channels, 3 * s->channels, dtype));
    bp->pk_proj = pad256(nystra::block_wpack_bytes(s->channels, s->channels, dtype));
    bp->bytes = 4 * bp->qkvo_bytes + bp->pk_qkv + bp->pk_proj;
    if (bp->variant == NYSTRA_VARIANT_SPLIT && bp->p.units > 0)
        bp->bytes += nystra::split_workspace_bytes(bp->p);
    return NYSTRA_OK;
}

// Bytes of the packed W_qkv and W_proj image (each part padded to 256 bytes;
// 0 when channels > 256).
size_t packed_parts(int C, int dtype, size_t *qkv_part)
{
    const size_t q = pad256(nystra::block_wpack_bytes(C, 3 * C, dtype));
    *qkv_part = q;
    return q + pad256(nystra::block_wpack_bytes(C, C, dtype));
}

// The block of nystra_block_forward.  With with_packed, the GEMMs read the
// weight image at `packed` (required when channels <= 256, ignored above)
// instead of packing W_qkv and W_proj into the workspace first.
int block_forward(const void *X, const void *Wqkv, const void *bqkv, const void *Wproj,
                  const void *bproj, bool with_packed, const void *packed,
                  size_t packed_bytes, void *Y,
                  const nystra_block_shape *shape, int m, int dtype, const nystra_opts *opts,
                  int attention, void *workspace, size_t workspace_bytes, void *stream)
{
    BlockPlan bp;
    int rc = plan_block(shape, m, dtype, opts, attention, &bp);
    if (rc != NYSTRA_OK)
        return rc;
    if (shape->batch == 0)
        return NYSTRA_OK;
    const bool use_packed = with_packed && bp.pk_qkv != 0;
    if (!X || !Wqkv || !Wproj || !Y || (use_packed && !packed))
        return NYSTRA_ERR_NULL;
    const int eb = dtype_bytes(dtype), C = shape->channels;
    if (misaligned(X, eb) || misaligned(Wqkv, eb) || misaligned(Wproj, eb) || misaligned(Y, eb) ||
        (bqkv && misaligned(bqkv, eb)) || (bproj && misaligned(bproj, eb)))
        return NYSTRA_ERR_ALIGN;
    const int64_t rows = int64_t(shape->batch) * shape->height * shape->width;
    const int64_t xb = rows * C * eb, wqb = int64_t(C) * 3 * C * eb, wpb = int64_t(C) * C * eb;
    if (overlaps(Y, xb, X, xb) || overlaps(Y, xb, Wqkv, wqb) || overlaps(Y, xb, Wproj, wpb) ||
        (bqkv && overlaps(Y, xb, bqkv, 3 * C * eb)) || (bproj && overlaps(Y, xb, bproj, C * eb)))
        return NYSTRA_ERR_OVERLAP;
    if (!workspace || workspace_bytes < bp.bytes || misaligned(workspace, 256))
        return NYSTRA_ERR_WORKSPACE;
    const int64_t wsb = int64_t(bp.bytes);
    if (overlaps(workspace, wsb, X, xb) || overlaps(workspace, wsb, Y, xb) ||
        overlaps(workspace, wsb, Wqkv, wqb) || overlaps(workspace, wsb, Wproj, wpb) ||
        (bqkv && overlaps(workspace, wsb, bqkv, 3 * C * eb)) ||
        (bproj && overlaps(workspace, wsb, bproj, C * eb)))
        return NYSTRA_ERR_WORKSPACE;
    if (use_packed) {   // read by the GEMMs only: no bytes shared with Y or the workspace
        const int64_t pb = int64_t(bp.pk_qkv + bp.pk_proj);
        if (packed_bytes < size_t(pb))
            return NYSTRA_ERR_WORKSPACE;
        if (misaligned(packed, 256))
            return NYSTRA_ERR_ALIGN;
        if (overlaps(packed, pb, Y, xb) || overlaps(packed, pb, workspace, wsb))
            return NYSTRA_ERR_OVERLAP;
    }
    char *ws = static_cast<char *>(workspace);
    void *q = ws, *k = ws + bp.qkvo_bytes, *v = ws + 2 * bp.qkvo_bytes,
         *o = ws + 3 * bp.qkvo_bytes;
    const char *pkq = nullptr, *pkp = nullptr;
    if (bp.pk_qkv) {
        pkq = use_packed ? static_cast<const char *>(packed) : ws + 4 * bp.qkvo_bytes;
        pkp = pkq + bp.pk_qkv;
    }
    char *attn_ws = ws + 4 * bp.qkvo_bytes + bp.pk_qkv + bp.pk_proj;
    hipStream_t st = static_cast<hipStream_t>(stream);
    clear_stale_error();
    if (pkq && !use_packed) {
        const hipError_t e = nystra::launch_block_wpack(Wqkv, Wproj, C, dtype,
                                                        const_cast<char *>(pkq),
                                                        const_cast<char *>(pkp), st);
        if (e != hipSuccess)
            return finish_launch(e);
    }
    nystra::BlockGemm g;
    g.rows = rows;
    g.H = shape->height;
    g.W = shape->width;
    g.C = C;
    g.heads = shape->heads;
    g.w = shape->window;
    g.shift = shape->shift;
    g.dtype = dtype;
    g.proj = false;
    g.a = X;
    g.wt = Wqkv;
    g.wpk = pkq;
    g.bias = bqkv;
    g.out0 = q;
    g.out1 = k;
    g.out2 = v;
    hipError_t e = nystra::launch_block_gemm(g, st);
    if (e != hipSuccess)
        return finish_launch(e);
    Problem p = bp.p;
    p.q = q;
    p.k = k;
    p.v = v;
    p.o = o;
    if (bp.variant == -1)
        e = nystra::launch_exact(p, st);
    else if (bp.variant == NYSTRA_VARIANT_SPLIT)
        e = nystra::launch_split(p, attn_ws, st);
    else if (bp.variant == NYSTRA_VARIANT_TILED && nystra::tiled_supported(p))
        e = nystra::launch_tiled_forward(p, st);
    else
        e = nystra::launch_generic_forward(p, st);
    if (e != hipSuccess)
        return finish_launch(e);
    g.proj = true;
    g.a = o;
    g.wt = Wproj;
    g.wpk = pkp;
    g.bias = bproj;
    g.out0 = Y;
    g.out1 = g.out2 = nullptr;
    return finish_launch(nystra::launch_block_gemm(g, st));
}


}  // namespace

extern "C" {

int nystra_block_workspace_size(const nystra_block_shape *shape, int m, int dtype,
                                const nystra_opts *opts, int attention, size_t *bytes)
{
    if (!bytes)
        return NYSTRA_ERR_NULL;
    BlockPlan bp;
    const int rc = plan_block(shape, m, dtype, opts, attention, &bp);
    if (rc != NYSTRA_OK)
        return rc;
    *bytes = shape->batch == 0 ? 0 : bp.bytes;
    return NYSTRA_OK;
}

int nystra_block_forward(const void *X, const void *Wqkv, const void *bqkv, const void *Wproj,
                         const void *bproj, void *Y, const nystra_block_shape *shape, int m,
                         int dtype, const nystra_opts *opts, int attention, void *workspace,
                         size_t workspace_bytes, void *stream)
{
    return block_forward(X, Wqkv, bqkv, Wproj, bproj, false, nullptr, 0, Y, shape, m, dtype,
                         opts, attention, workspace, workspace_bytes, stream);
}

int nystra_block_packed_size(int channels, int dtype, size_t *bytes)
{
    if (!bytes)
        return NYSTRA_ERR_NULL;
    if (dtype != NYSTRA_F32 && dtype != NYSTRA_BF16)
        return NYSTRA_ERR_DTYPE;
    if (channels < 1 || channels > 4096)
        return NYSTRA_ERR_SHAPE;
    size_t q;
    *bytes = packed_parts(channels, dtype, &q);
    return NYSTRA_OK;
}

int nystra_block_pack_weights(const void *Wqkv, const void *Wproj, int channels, int dtype,
                              void *packed, size_t packed_bytes, void *stream)
{
    size_t q = 0, need = 0;
    const int rc = nystra_block_packed_size(channels, dtype, &need);
    if (rc != NYSTRA_OK)
        return rc;
    if (need == 0)
        return NYSTRA_OK;   // channels > 256: the block reads the weights as given
    if (!Wqkv || !Wproj || !packed)
        return NYSTRA_ERR_NULL;
    const int eb = dtype_bytes(dtype);
    if (misaligned(Wqkv, eb) || misaligned(Wproj, eb) || misaligned(packed, 256))
        return NYSTRA_ERR_ALIGN;
    if (packed_bytes < need)
        return NYSTRA_ERR_WORKSPACE;
    const int64_t C = channels;
    if (overlaps(packed, int64_t(need), Wqkv, C * 3 * C * eb) ||
        overlaps(packed, int64_t(need), Wproj, C * C * eb))
        return NYSTRA_ERR_OVERLAP;
    packed_parts(channels, dtype, &q);
    char *pk = static_cast<char *>(packed);
    clear_stale_error();
    return finish_launch(nystra::launch_block_wpack(Wqkv, Wproj, channels, dtype, pk, pk + q,
                                                    static_cast<hipStream_t>(stream)));
}

int nystra_block_forward_packed(const void *X, const void *Wqkv, const void *bqkv,
                                const void *Wproj, const void *bproj, const void *packed,
                                size_t packed_bytes, void *Y, const nystra_block_shape *shape,
                                int m, int dtype, const nystra_opts *opts, int attention,
                                void *workspace, size_t workspace_bytes, void *stream)
{
    return block_forward(X, Wqkv, bqkv, Wproj, bproj, true, packed, packed_bytes, Y, shape, m,
                         dtype, opts, attention, workspace, workspace_bytes, stream);
}

const char *nystra_status_str(int status)
{
    switch (status) {
    case NYSTRA_OK: return "ok";
    case NYSTRA_ERR_NULL: return "null pointer";
    case NYSTRA_ERR_SHAPE: return "shape out of range or no pooling grid";
    case NYSTRA_ERR_DTYPE: return "unsupported dtype";
    case NYSTRA_ERR_ALIGN: return "misaligned pointer";
    case NYSTRA_ERR_OVERLAP: return "output overlaps an input";
    case NYSTRA_ERR_UNSUPPORTED: return "forced kernel variant cannot run this shape";
    case NYSTRA_ERR_HIP: return "HIP launch error";
    case NYSTRA_ERR_ARG: return "invalid argument";
    case NYSTRA_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    default: return "unknown status";
    }
}

const char *nystra_last_error(void) { return g_last_error; }

}  // extern "C"
