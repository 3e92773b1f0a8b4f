// Portable PnP-Nystra kernels: one 256-thread workgroup per (window, head)
// unit, every shape within the library limits (N <= 2^20, d_h <= 128, m <= 64),
// fp32 vector arithmetic, LDS for the small per-unit matrices.  They are the
// fallback behind the MFMA-tiled kernels and the reference the tiled kernels
// are compared against on shapes both cover.
#include "device_common.hpp"
#include "internal.hpp"

namespace nystra {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

// Step 1 (Sec. 2.2): mean of the tokens of landmark l's pooling patch, for
// every (l, c) pair handled by this thread.  Writes fp32 [m][d] to dst.
template <class E>
__device__ void pool_unit(const typename E::T *x, float *dst, const Geometry &g, int m, int d,
                          int tid, int nthreads)
{
    const float inv = 1.0f / float(g.pr * g.pc);
    for (int idx = tid; idx < m * d; idx += nthreads) {
        const int l = idx / d, c = idx - (idx / d) * d;
        const int r0 = (l / g.gc) * g.pr, c0 = (l % g.gc) * g.pc;
        float acc = 0.f;
        for (int r = r0; r < r0 + g.pr; ++r)
            for (int cc = c0; cc < c0 + g.pc; ++cc)
                acc += E::load(x, int64_t(r * g.cols + cc) * d + c);
        dst[idx] = acc * inv;
    }
}

template <class E>
__global__ void __launch_bounds__(kThreads)
landmark_pool_kernel(const typename E::T *__restrict__ q, const typename E::T *__restrict__ k,
                     float *__restrict__ qbar, float *__restrict__ kbar,
                     int32_t *__restrict__ map, int N, int d, int m, Geometry g)
{
    const int64_t u = blockIdx.x;
    const int64_t in_off = u * int64_t(N) * d;
    const int64_t out_off = u * int64_t(m) * d;
    pool_unit<E>(q + in_off, qbar + out_off, g, m, d, threadIdx.x, kThreads);
    pool_unit<E>(k + in_off, kbar + out_off, g, m, d, threadIdx.x, kThreads);
    if (map != nullptr && u == 0) {
        for (int t = threadIdx.x; t < N; t += kThreads) {
            const int r = t / g.cols, c = t % g.cols;
            map[t] = (r / g.pr) * g.gc + c / g.pc;
        }
    }
}

// LDS carve-up of the generic forward kernel (floats).  Qbar and m_U are
// dead once A is formed, so Z, X, Y and Y2 take their place; W = Z T is
// written over X, Y and Y2 after the iteration (or past them when it is
// longer).  At m = 64, d_h = 128 the workgroup takes 148 KB.
struct Lds {
    int kbar, qbar, mu, t, w, a, z, x, y, y2, norms, total;
    __host__ __device__ Lds(int m, int d)
    {
        int o = 0;
        kbar = o; o += m * d;
        t = o;    o += m * (d + 1);
        a = o;    o += m * m;
        const int r = o;   // Qbar and m_U, then Z, X, Y, Y2 and W
        qbar = r;
        mu = r + m * d;
        z = r;
        x = z + m * m;
        y = x + m * m;
        y2 = y + m * m;
        w = x;
        const int wend = w + m * (d + 1), yend = y2 + m * m;
        o = wend > yend ? wend : yend;
        norms = o; o += 2 * m + 1;
        total = o;
    }
};

// out (n x p) = L (n x k) * R (k x p), all row-major in LDS; block-wide.
__device__ void lds_matmul(const float *L, const float *R, float *out, int n, int kk, int p)
{
    for (int idx = threadIdx.x; idx < n * p; idx += kThreads) {
        const int i = idx / p, j = idx - (idx / p) * p;
        float acc = 0.f;
        for (int q = 0; q < kk; ++q)
            acc = fmaf(L[i * kk + q], R[q * p + j], acc);
        out[idx] = acc;
    }
}

// dst = c I - src  (m x m), block-wide.
__device__ void shift_neg(const float *src, float *dst, int m, float c)
{
    for (int idx = threadIdx.x; idx < m * m; idx += kThreads) {
        const int i = idx / m, j = idx - (idx / m) * m;
        dst[idx] = (i == j ? c : 0.f) - src[idx];
    }
}

// DM bounds d_h (64 or 128): the per-thread feature arrays are sized by it.
template <class E, int DM>
__global__ void __launch_bounds__(kThreads)
generic_forward_kernel(const typename E::T *__restrict__ q, const typename E::T *__restrict__ k,
                       const typename E::T *__restrict__ v, typename E::T *__restrict__ o,
                       int N, int d, int m, int iters, float scale, Geometry g)
{
    extern __shared__ float lds[];
    const Lds L(m, d);
    float *kbar = lds + L.kbar, *qbar = lds + L.qbar, *mu = lds + L.mu;
    float *T = lds + L.t, *Wm = lds + L.w;
    float *A = lds + L.a, *Z = lds + L.z, *X = lds + L.x, *Y = lds + L.y, *Y2 = lds + L.y2;
    float *norms = lds + L.norms;

    const int64_t base = int64_t(blockIdx.x) * N * d;
    const typename E::T *qu = q + base, *ku = k + base, *vu = v + base;
    typename E::T *ou = o + base;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float s2 = scale * kLog2e;   // logits carried in base-2 units

    constexpr int kMaxD = DM;
    // Step 1: landmarks.
    pool_unit<E>(qu, qbar, g, m, d, tid, kThreads);
    pool_unit<E>(ku, kbar, g, m, d, tid, kThreads);
    __syncthreads();

    // Step 3 (G_U side): m_U(l) = max_t s qbar_l . k_t, then
    // T = G_U^n [V | 1] with G_U^n = exp(s qbar K^T - m_U).
    for (int l = wave; l < m; l += kWaves) {
        float mx = -INFINITY;
        for (int t = lane; t < N; t += 64) {
            float acc = 0.f;
            for (int c = 0; c < d; ++c)
                acc = fmaf(qbar[l * d + c], E::load(ku, int64_t(t) * d + c), acc);
            mx = fmaxf(mx, acc * s2);
        }
        mx = wave_max(mx);
        float tacc[kMaxD + 1];
#pragma unroll
        for (int c = 0; c <= kMaxD; ++c)
            tacc[c] = 0.f;
        for (int t = lane; t < N; t += 64) {
            float acc = 0.f;
            for (int c = 0; c < d; ++c)
                acc = fmaf(qbar[l * d + c], E::load(ku, int64_t(t) * d + c), acc);
            const float e = exp2f(acc * s2 - mx);
#pragma unroll
            for (int c = 0; c < kMaxD; ++c)
                if (c < d)
                    tacc[c] = fmaf(e, E::load(vu, int64_t(t) * d + c), tacc[c]);
            tacc[kMaxD] += e;
        }
#pragma unroll
        for (int c = 0; c < kMaxD; ++c)
            if (c < d) {
                const float r = wave_sum(tacc[c]);
                if (lane == 0)
                    T[l * (d + 1) + c] = r;
            }
        const float r = wave_sum(tacc[kMaxD]);
        if (lane == 0) {
            T[l * (d + 1) + d] = r;
            mu[l] = mx;
        }
    }
    __syncthreads();

    // Step 2, normalised: A = G_A^n = exp(s qbar kbar^T - m_U) (rows by m_U).
    for (int idx = tid; idx < m * m; idx += kThreads) {
        const int i = idx / m, j = idx - (idx / m) * m;
        float acc = 0.f;
        for (int c = 0; c < d; ++c)
            acc = fmaf(qbar[i * d + c], kbar[j * d + c], acc);
        A[idx] = exp2f(acc * s2 - mu[i]);
    }
    __syncthreads();   // Qbar and m_U dead from here (Z, X, Y, Y2 take their place)

    // Step 4: Z_0 = A^T / (||A||_1 ||A||_inf), then the iteration.
    for (int i = tid; i < m; i += kThreads) {
        float rs = 0.f, cs = 0.f;
        for (int j = 0; j < m; ++j) {
            rs += fabsf(A[i * m + j]);
            cs += fabsf(A[j * m + i]);
        }
        norms[i] = rs;
        norms[m + i] = cs;
    }
    __syncthreads();
    if (tid == 0) {
        float ninf = 0.f, n1 = 0.f;
        for (int i = 0; i < m; ++i) {
            ninf = fmaxf(ninf, norms[i]);
            n1 = fmaxf(n1, norms[m + i]);
        }
        norms[2 * m] = 1.0f / (n1 * ninf);
    }
    __syncthreads();
    const float alpha = norms[2 * m];
    for (int idx = tid; idx < m * m; idx += kThreads) {
        const int i = idx / m, j = idx - (idx / m) * m;
        Z[idx] = alpha * A[j * m + i];
    }
    __syncthreads();
    for (int it = 0; it < iters; ++it) {
        lds_matmul(A, Z, X, m, m, m);       // X = A Z
        __syncthreads();
        shift_neg(X, Y, m, 7.f);            // Y = 7I - X
        __syncthreads();
        lds_matmul(X, Y, Y2, m, m, m);      // Y2 = X (7I - X)
        __syncthreads();
        shift_neg(Y2, Y, m, 15.f);          // Y = 15I - Y2
        __syncthreads();
        lds_matmul(X, Y, Y2, m, m, m);      // Y2 = X (15I - ...)
        __syncthreads();
        shift_neg(Y2, Y, m, 13.f);          // Y = 13I - Y2
        __syncthreads();
        lds_matmul(Z, Y, Y2, m, m, m);      // Y2 = Z (13I - ...)
        __syncthreads();
        for (int idx = tid; idx < m * m; idx += kThreads)
            Z[idx] = 0.25f * Y2[idx];
        __syncthreads();
    }

    // Steps 5-6 re-associated: W = Z T  (m x (d+1)).
    lds_matmul(Z, T, Wm, m, m, d + 1);
    __syncthreads();

    // Steps 3 (G_L side), 6 and 7 per token: G_L^n row, O_N, O_D, divide.
    for (int t = tid; t < N; t += kThreads) {
        float qv[kMaxD];
#pragma unroll
        for (int c = 0; c < kMaxD; ++c)
            qv[c] = c < d ? E::load(qu, int64_t(t) * d + c) : 0.f;
        float mx = -INFINITY;
        for (int j = 0; j < m; ++j) {
            float acc = 0.f;
#pragma unroll
            for (int c = 0; c < kMaxD; ++c)
                if (c < d)
                    acc = fmaf(qv[c], kbar[j * d + c], acc);
            mx = fmaxf(mx, acc * s2);
        }
        float on[kMaxD + 1];
#pragma unroll
        for (int c = 0; c <= kMaxD; ++c)
            on[c] = 0.f;
        for (int j = 0; j < m; ++j) {
            float acc = 0.f;
#pragma unroll
            for (int c = 0; c < kMaxD; ++c)
                if (c < d)
                    acc = fmaf(qv[c], kbar[j * d + c], acc);
            const float e = exp2f(acc * s2 - mx);
#pragma unroll
            for (int c = 0; c < kMaxD; ++c)
                if (c < d)
                    on[c] = fmaf(e, Wm[j * (d + 1) + c], on[c]);
            on[kMaxD] = fmaf(e, Wm[j * (d + 1) + d], on[kMaxD]);
        }
        const float inv = 1.0f / on[kMaxD];
#pragma unroll
        for (int c = 0; c < kMaxD; ++c)
            if (c < d)
                E::store(ou, int64_t(t) * d + c, on[c] * inv);
    }
}

template <class E, int DM>
hipError_t launch_generic_t(const Problem &p, hipStream_t stream)
{
    const Lds L(p.m, p.d);
    const size_t lds_bytes = size_t(L.total) * sizeof(float);
    hipLaunchKernelGGL((generic_forward_kernel<E, DM>), dim3(unsigned(p.units)), dim3(kThreads),
                       lds_bytes, stream, static_cast<const typename E::T *>(p.q),
                       static_cast<const typename E::T *>(p.k),
                       static_cast<const typename E::T *>(p.v),
                       static_cast<typename E::T *>(p.o), p.N, p.d, p.m, p.iters, p.scale,
                       p.geo);
    return hipGetLastError();
}

}  // namespace

size_t generic_lds_bytes(int m, int d) { return size_t(Lds(m, d).total) * sizeof(float); }

hipError_t launch_generic_forward(const Problem &p, hipStream_t stream)
{
    if (p.d <= 64)
        return p.dtype == 0 ? launch_generic_t<F32, 64>(p, stream)
                            : launch_generic_t<BF16, 64>(p, stream);
    return p.dtype == 0 ? launch_generic_t<F32, 128>(p, stream)
                        : launch_generic_t<BF16, 128>(p, stream);
}

hipError_t launch_landmark_pool(const Problem &p, float *qbar, float *kbar, int32_t *map,
                                hipStream_t stream)
{
    if (p.dtype == 0)
        hipLaunchKernelGGL(landmark_pool_kernel<F32>, dim3(unsigned(p.units)), dim3(kThreads), 0,
                           stream, static_cast<const float *>(p.q),
                           static_cast<const float *>(p.k), qbar, kbar, map, p.N, p.d, p.m,
                           p.geo);
    else
        hipLaunchKernelGGL(landmark_pool_kernel<BF16>, dim3(unsigned(p.units)), dim3(kThreads),
                           0, stream, static_cast<const uint16_t *>(p.q),
                           static_cast<const uint16_t *>(p.k), qbar, kbar, map, p.N, p.d, p.m,
                           p.geo);
    return hipGetLastError();
}

}  // namespace nystra
