// Exact windowed softmax self-attention, Eq. (1): O = softmax(s Q K^T) V per
// (window, head) unit, with the row maximum subtracted inside the softmax
// (kept as a running maximum over key blocks).  This is the comparison
// baseline for the Nystrom kernels.
#include "device_common.hpp"
#include "internal.hpp"

namespace nystra {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxD = 64;
constexpr int kKeyTile = 64;   // keys staged in LDS per step

// One thread per query row; keys and values of the unit are staged through
// LDS in tiles of kKeyTile rows shared by the whole workgroup.
template <class E>
__global__ void __launch_bounds__(kThreads)
exact_rows_kernel(const typename E::T *__restrict__ q, const typename E::T *__restrict__ k,
                  const typename E::T *__restrict__ v, typename E::T *__restrict__ o,
                  int N, int d, float scale)
{
    __shared__ float ks[kKeyTile * kMaxD];
    __shared__ float vs[kKeyTile * kMaxD];
    const int64_t base = int64_t(blockIdx.x) * N * d;
    const int row = blockIdx.y * kThreads + threadIdx.x;
    const bool active = row < N;
    const float s2 = scale * kLog2e;

    float qv[kMaxD], acc[kMaxD];
#pragma unroll
    for (int c = 0; c < kMaxD; ++c) {
        qv[c] = (active && c < d) ? E::load(q + base, int64_t(row) * d + c) * s2 : 0.f;
        acc[c] = 0.f;
    }
    float mrun = -INFINITY, lsum = 0.f;

    for (int t0 = 0; t0 < N; t0 += kKeyTile) {
        const int nt = min(kKeyTile, N - t0);
        __syncthreads();
        for (int idx = threadIdx.x; idx < nt * d; idx += kThreads) {
            const int tt = idx / d, c = idx - (idx / d) * d;
            ks[tt * kMaxD + c] = E::load(k + base, int64_t(t0 + tt) * d + c);
            vs[tt * kMaxD + c] = E::load(v + base, int64_t(t0 + tt) * d + c);
        }
        __syncthreads();
        if (!active)
            continue;
        for (int tt = 0; tt < nt; ++tt) {
            float a = 0.f;
#pragma unroll
            for (int c = 0; c < kMaxD; ++c)
                if (c < d)
                    a = fmaf(qv[c], ks[tt * kMaxD + c], a);
            if (a > mrun) {
                const float r = exp2f(mrun - a);
                lsum *= r;
#pragma unroll
                for (int c = 0; c < kMaxD; ++c)
                    acc[c] *= r;
                mrun = a;
            }
            const float p = exp2f(a - mrun);
            lsum += p;
#pragma unroll
            for (int c = 0; c < kMaxD; ++c)
                if (c < d)
                    acc[c] = fmaf(p, vs[tt * kMaxD + c], acc[c]);
        }
    }
    if (active) {
        const float inv = 1.0f / lsum;
#pragma unroll
        for (int c = 0; c < kMaxD; ++c)
            if (c < d)
                E::store(o + base, int64_t(row) * d + c, acc[c] * inv);
    }
}

template <class E>
hipError_t launch_exact_t(const Problem &p, hipStream_t stream)
{
    const dim3 grid(unsigned(p.units), unsigned((p.N + kThreads - 1) / kThreads));
    hipLaunchKernelGGL(exact_rows_kernel<E>, grid, dim3(kThreads), 0, stream,
                       static_cast<const typename E::T *>(p.q),
                       static_cast<const typename E::T *>(p.k),
                       static_cast<const typename E::T *>(p.v),
                       static_cast<typename E::T *>(p.o), p.N, p.d, p.scale);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_exact(const Problem &p, hipStream_t stream)
{
    return p.dtype == 0 ? launch_exact_t<F32>(p, stream) : launch_exact_t<BF16>(p, stream);
}

}  // namespace nystra
