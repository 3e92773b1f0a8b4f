// Exact windowed softmax self-attention, Eq. (1): O = softmax(s Q K^T) V per
// (window, head) unit, with the row maximum subtracted inside the softmax
// (kept as a running maximum over key blocks).  This is the comparison
// baseline for the Nystrom kernels.
//
// exact_tiled_kernel (N % 32 == 0, d_h in the tiled widths): flash-style.
// One wavefront owns 16 queries and walks the keys in blocks of 32.  Scores
// are produced transposed, S^T = K Q^T, so each lane column is one query and
// the running max / sum / rescale stay in the lane; the output is accumulated
// transposed as well, O^T += V^T P^T.  fp32 inputs use the fp32 matrix cores;
// bf16 inputs use v_mfma_f32_16x16x32_bf16 for both products with P rounded
// to bf16 (V is staged transposed in LDS for the second product).
// exact_rows_kernel: one thread per query row, any shape.
#include "internal.hpp"
#include "tile_common.hpp"

namespace nystra {
namespace {

constexpr int kThreads = 256;

// One thread per query row; keys and values of the unit are staged through
// LDS in tiles of kKeyTile rows shared by the whole workgroup.  DM bounds d_h
// (64 or 128; the per-thread rows are sized by it).
template <class E, int DM>
__global__ void __launch_bounds__(kThreads)
exact_rows_kernel(const typename E::T *__restrict__ q, const typename E::T *__restrict__ k,
                  const typename E::T *__restrict__ v, typename E::T *__restrict__ o,
                  int N, int d, float scale)
{
    constexpr int kMaxD = DM;
    constexpr int kKeyTile = 4096 / DM;   // keys staged in LDS per step (32 KB)
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

using namespace tile;

// Eight features of one row as raw bf16 pairs (slots outside the lane
// group's chunk zeroed; see load_chunk8).  D is even, so invalid slots come
// in whole 32-bit pairs.
template <int D>
__device__ inline U16B load_chunk8_raw(const uint16_t *row, int g)
{
    U16B u = *reinterpret_cast<const U16B *>(row + chunk_start<D>(g));
#pragma unroll
    for (int j = 0; j < 4; ++j)
        if (!slot_valid<D>(g, 2 * j))
            u.w[j] = 0u;
    return u;
}

__device__ inline bf8 as_bf8(const U16B &u) { return __builtin_bit_cast(bf8, u); }

// Two probabilities (finite, in [0, 1]) as a bf16 pair, rounded to nearest
// even by the conversion instruction.
__device__ inline uint32_t pack_bf16(float lo, float hi) { return cvt_bf16x2(lo, hi); }

constexpr int kExactWaves = 4;

template <class E, int D, bool BF>
__global__ void __launch_bounds__(64 * kExactWaves)
exact_tiled_kernel(const typename E::T *__restrict__ q, const typename E::T *__restrict__ k,
                   const typename E::T *__restrict__ v, typename E::T *__restrict__ o, int N,
                   float s2, int qblocks)
{
    extern __shared__ uint16_t vt[];   // bf16 only: V^T, [32 features][N + 8 keys]
    constexpr int d = D;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int g = lane >> 4, c = lane & 15;
    const int64_t unit = blockIdx.x / qblocks;
    const int NT = N >> 4, pitch = N + 8;
    const int qt = (blockIdx.x % qblocks) * kExactWaves + wave;   // query tile of this wave
    const int64_t base = unit * int64_t(N) * d;
    const typename E::T *qu = q + base, *ku = k + base, *vu = v + base;
    typename E::T *ou = o + base;
    constexpr bool bf = BF;   // bf16 inputs on the bf16 matrix cores

    if constexpr (bf) {
        for (int kt = wave; kt < NT; kt += kExactWaves) {
            const U16B u = load_chunk8_raw<D>(
                reinterpret_cast<const uint16_t *>(vu) + int64_t(16 * kt + c) * d, g);
#pragma unroll
            for (int s = 0; s < 8; ++s)
                if (slot_valid<D>(g, s))
                    vt[(chunk_start<D>(g) + s) * pitch + 16 * kt + c] =
                        uint16_t(u.w[s >> 1] >> (16 * (s & 1)));
        }
        __syncthreads();
    }
    if (qt >= NT)
        return;   // after the only block-level barrier

    const int qrow = 16 * qt + c;
    float qf[8];
    U16B qraw;
    if constexpr (bf)
        qraw = load_chunk8_raw<D>(reinterpret_cast<const uint16_t *>(qu) + int64_t(qrow) * d, g);
    else
        load_chunk8<E, D>(qu + int64_t(qrow) * d, g, qf);

    float mrun = -INFINITY, lrun = 0.f;
    f4 OT[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};   // O^T[16ct+4g+i][query c]
    for (int kb = 0; kb < NT; kb += 2) {
        f4 S[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int key = 16 * (kb + h) + c;
            f4 acc = {0.f, 0.f, 0.f, 0.f};
            if constexpr (bf) {
                const U16B kraw = load_chunk8_raw<D>(
                    reinterpret_cast<const uint16_t *>(ku) + int64_t(key) * d, g);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf8(kraw), as_bf8(qraw), acc, 0,
                                                             0, 0);
            } else {
                float kf[8];
                load_chunk8<E, D>(ku + int64_t(key) * d, g, kf);
#pragma unroll
                for (int s = 0; s < 8; ++s)
                    acc = mfma4(kf[s], qf[s], acc);
            }
            S[h] = acc;   // lane (g,c): S[query c][key 16(kb+h) + 4g + i]
        }
        float bmax = fmaxf(fmaxf(fmaxf(S[0][0], S[0][1]), fmaxf(S[0][2], S[0][3])),
                           fmaxf(fmaxf(S[1][0], S[1][1]), fmaxf(S[1][2], S[1][3])));
        const float mnew = fmaxf(mrun, s2 * max_groups(bmax));
        const float sc = fast_exp2(mrun - mnew);
        float psum = 0.f;
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                S[h][i] = fast_exp2(fmaf(s2, S[h][i], -mnew));
                psum += S[h][i];
            }
        lrun = fmaf(lrun, sc, sum_groups(psum));
        mrun = mnew;
#pragma unroll
        for (int ct = 0; ct < 2; ++ct) {
            f4 upd;
            if constexpr (bf) {
                // A = V^T rows (feature 16ct+c), keys {4g..4g+3} of both tiles;
                // B = P^T for the same keys.
                const uint16_t *row = vt + (16 * ct + c) * pitch + 16 * kb + 4 * g;
                const uint2 v0 = *reinterpret_cast<const uint2 *>(row);
                const uint2 v1 = *reinterpret_cast<const uint2 *>(row + 16);
                U16B a, b;
                a.w[0] = v0.x; a.w[1] = v0.y; a.w[2] = v1.x; a.w[3] = v1.y;
                b.w[0] = pack_bf16(S[0][0], S[0][1]);
                b.w[1] = pack_bf16(S[0][2], S[0][3]);
                b.w[2] = pack_bf16(S[1][0], S[1][1]);
                b.w[3] = pack_bf16(S[1][2], S[1][3]);
                upd = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf8(a), as_bf8(b),
                                                             f4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
            } else {
                // LT = V tile in D-layout: V[key 16(kb+h) + 4g + i][feature 16ct + c].
                const int f = 16 * ct + c;
                upd = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    f4 vd;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float x = E::load(vu, int64_t(16 * (kb + h) + 4 * g + i) * d +
                                                        min(f, d - 1));
                        vd[i] = f < d ? x : 0.f;
                    }
                    upd += mm16(vd, S[h]);
                }
            }
            OT[ct] = OT[ct] * sc + upd;
        }
    }
    const float inv = __builtin_amdgcn_rcpf(lrun);
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int f = 16 * ct + 4 * g + i;
            if (f < d)
                E::store(ou, int64_t(qrow) * d + f, OT[ct][i] * inv);
        }
}

// ---- bf16, N a multiple of 64: key blocks streamed through LDS -------------
//
// A workgroup of NW waves covers 16 QT NW queries of one unit; wave w owns QT
// query tiles and keeps their output, transposed, in registers.  The unit's
// keys are streamed in blocks of 64 through two LDS buffers -- K rows, and V
// transposed -- so every key and value is read from memory once per
// workgroup; the next block is requested before the current one is computed.
// Per block and query tile: S^T = K Q^T (one 16x16x32 bf16 product per key
// tile), probabilities exp(s q.k - m) rounded to bf16 for O^T += V^T P^T (as
// bf16 flash attention does), the row sums accumulated in fp32 from the
// unrounded probabilities.
//
// The reference point m of a query's exponentials only grows, and only when a
// score exceeds it by more than 2^8 (base 2): then it becomes the running
// maximum over the four lane groups and the accumulated sums are rescaled.
// Every probability thus stays in (0, 2^8], and the quotient of Eq. (1) is
// the same for any reference point; only the rounding differs, and the bf16
// rounding of a probability stays relative (at most 2^-8 of it).

constexpr int kXB = 64;         // keys per block
constexpr int kXKP = 40;        // pitch (bf16) of the K rows in LDS
constexpr int kXVP = kXB + 8;   // pitch (bf16) of the V^T rows in LDS

template <int D>
struct XBufs {
    static constexpr int kbytes = kXB * kXKP * 2;
    static constexpr int vbytes = 32 * kXVP * 2;
    static constexpr int bytes = kbytes + vbytes;   // one buffer
};

template <int D, int QT>
__global__ void __launch_bounds__(512)
exact_blocked_kernel(const uint16_t *__restrict__ q, const uint16_t *__restrict__ k,
                     const uint16_t *__restrict__ v, uint16_t *__restrict__ o, int N, float s2,
                     int wpu)
{
    constexpr int NCT = (D + 15) / 16;
    using X = XBufs<D>;
    extern __shared__ __attribute__((aligned(16))) unsigned char xsm[];
    const int nw = blockDim.x >> 6;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int g = lane >> 4, c = lane & 15;
    const int64_t unit = blockIdx.x / wpu;
    const int wg = int(blockIdx.x - unit * wpu);
    const int64_t base = unit * int64_t(N) * D;
    const uint16_t *qu = q + base, *ku = k + base, *vu = v + base;
    uint16_t *ou = o + base;
    const int q0 = (wg * nw + w) * 16 * QT;   // first query of this wave

    // V^T rows past D are zero (both buffers, never overwritten by the
    // staging below).  The row sums are fp32 sums of the unrounded
    // probabilities, as in the one-row reference, not a ones column of V
    // (which would sum the bf16-rounded ones).
    if constexpr (16 * NCT > D) {
        constexpr int kPad = (16 * NCT - D) * kXB;
        for (int idx = threadIdx.x; idx < 2 * kPad; idx += blockDim.x) {
            const int b = idx / kPad, r = idx % kPad;
            const int f = D + r / kXB, key = r % kXB;
            uint16_t *vt = reinterpret_cast<uint16_t *>(xsm + b * X::bytes + X::kbytes);
            vt[f * kXVP + key] = uint16_t(0);
        }
    }
    // Staging: thread t of the first 256 (a workgroup has at least four
    // waves) takes key t / 4 of the block, chunk t % 4 (the slot layout of
    // load_chunk8), of both K and V.
    const bool stager = threadIdx.x < 256;
    const int skey = (threadIdx.x >> 2) & 63, sg = threadIdx.x & 3;
    U16B kst, vst;
    auto fetch = [&](int blk) {
        if (stager) {
            const int64_t row = int64_t(blk * kXB + skey) * D + chunk_start<D>(sg);
            kst = *reinterpret_cast<const U16B *>(ku + row);
            vst = *reinterpret_cast<const U16B *>(vu + row);
        }
    };
    auto store = [&](int buf) {
        if (stager) {
            unsigned char *bb = xsm + buf * X::bytes;
            U16B kk = kst;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (!slot_valid<D>(sg, 2 * j))
                    kk.w[j] = 0u;
            *reinterpret_cast<U16B *>(bb + (skey * kXKP + 8 * sg) * 2) = kk;
            uint16_t *vt = reinterpret_cast<uint16_t *>(bb + X::kbytes);
#pragma unroll
            for (int x = 0; x < 8; ++x)
                if (slot_valid<D>(sg, x))
                    vt[(chunk_start<D>(sg) + x) * kXVP + skey] =
                        uint16_t(vst.w[x >> 1] >> (16 * (x & 1)));
        }
    };

    // This wave's query tiles in the slot layout, raw bf16.
    bf8 qf[QT];
#pragma unroll
    for (int t = 0; t < QT; ++t) {
        U16B u = *reinterpret_cast<const U16B *>(qu + int64_t(q0 + 16 * t + c) * D +
                                                 chunk_start<D>(g));
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (!slot_valid<D>(g, 2 * j))
                u.w[j] = 0u;
        qf[t] = __builtin_bit_cast(bf8, u);
    }
    f4 OT[QT][NCT];   // O^T[feature 16ct+4g+i][query q0+16t+c]
    float mref[QT], lsum[QT];
#pragma unroll
    for (int t = 0; t < QT; ++t) {
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
            OT[t][ct] = f4{0.f, 0.f, 0.f, 0.f};
        mref[t] = -INFINITY;
        lsum[t] = 0.f;
    }

    const int nblk = N / kXB;
    fetch(0);
    store(0);
    __syncthreads();
    for (int blk = 0; blk < nblk; ++blk) {
        const int buf = blk & 1;
        if (blk + 1 < nblk)
            fetch(blk + 1);   // in flight while this block is computed
        const unsigned char *bb = xsm + buf * X::bytes;
        bf8 kf[4];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
            kf[kt] = *reinterpret_cast<const bf8 *>(bb + ((16 * kt + c) * kXKP + 8 * g) * 2);
        // A operands of the value product: V^T rows 16ct+c, keys {4g..4g+3}
        // of the tiles 2kp and 2kp+1 (the k order of the probabilities below).
        bf8 vf[2][NCT];
        const uint16_t *vt = reinterpret_cast<const uint16_t *>(bb + X::kbytes);
#pragma unroll
        for (int kp = 0; kp < 2; ++kp)
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                const uint16_t *row = vt + (16 * ct + c) * kXVP + 32 * kp + 4 * g;
                const uint2 a0 = *reinterpret_cast<const uint2 *>(row);
                const uint2 a1 = *reinterpret_cast<const uint2 *>(row + 16);
                U16B u;
                u.w[0] = a0.x; u.w[1] = a0.y; u.w[2] = a1.x; u.w[3] = a1.y;
                vf[kp][ct] = __builtin_bit_cast(bf8, u);
            }
#pragma unroll
        for (int t = 0; t < QT; ++t) {
            f4 st[4];   // lane (g,c): S^T[key 16kt+4g+i][query q0+16t+c]
            float lmax = -INFINITY;
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) {
                st[kt] = mfma_bf16(kf[kt], qf[t], f4{0.f, 0.f, 0.f, 0.f});
                lmax = fmaxf(lmax, fmaxf(fmaxf(st[kt][0], st[kt][1]), fmaxf(st[kt][2], st[kt][3])));
            }
            if (__builtin_amdgcn_ballot_w64(s2 * lmax > mref[t] + 8.f) != 0) {
                const float mnew = fmaxf(mref[t], s2 * max_groups(lmax));
                const float f = fast_exp2(mref[t] - mnew);   // 0 on the first block
                lsum[t] *= f;
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
                    OT[t][ct] *= f;
                mref[t] = mnew;
            }
#pragma unroll
            for (int kt = 0; kt < 4; ++kt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    st[kt][i] = fast_exp2(fmaf(s2, st[kt][i], -mref[t]));
                    lsum[t] += st[kt][i];
                }
#pragma unroll
            for (int kp = 0; kp < 2; ++kp) {
                U16B pb;
                pb.w[0] = cvt_bf16x2(st[2 * kp][0], st[2 * kp][1]);
                pb.w[1] = cvt_bf16x2(st[2 * kp][2], st[2 * kp][3]);
                pb.w[2] = cvt_bf16x2(st[2 * kp + 1][0], st[2 * kp + 1][1]);
                pb.w[3] = cvt_bf16x2(st[2 * kp + 1][2], st[2 * kp + 1][3]);
                const bf8 pv = __builtin_bit_cast(bf8, pb);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
                    OT[t][ct] = mfma_bf16(vf[kp][ct], pv, OT[t][ct]);
            }
        }
        if (blk + 1 < nblk)
            store(buf ^ 1);
        __syncthreads();
    }

    // Divide by the row sums and store rows of O.
#pragma unroll
    for (int t = 0; t < QT; ++t) {
        const float inv = __builtin_amdgcn_rcpf(sum_groups(lsum[t]));
        uint16_t *orow = ou + int64_t(q0 + 16 * t + c) * D;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
            const int f = 16 * ct + 4 * g;
            const uint32_t p01 = cvt_bf16x2(OT[t][ct][0] * inv, OT[t][ct][1] * inv);
            const uint32_t p23 = cvt_bf16x2(OT[t][ct][2] * inv, OT[t][ct][3] * inv);
            if (f + 1 < D)
                *reinterpret_cast<uint32_t *>(orow + f) = p01;
            if (f + 3 < D)
                *reinterpret_cast<uint32_t *>(orow + f + 2) = p23;
        }
    }
}

// ---- fp32, N a multiple of 64: the same blocked structure on the fp32 matrix
// cores.  K rows and V^T are staged as fp32; S^T tiles are eight-step
// 16x16x4 products over the feature slots (the slot layout of load_chunk8);
// the probabilities stay fp32 and feed O^T += V^T P^T directly in the
// D-layout, with V^T read as the transposed left operand.

constexpr int kFKP = 36;        // pitch (floats) of the K rows in LDS
constexpr int kFVP = kXB + 4;   // pitch (floats) of the V^T rows in LDS

struct FBufs {
    static constexpr int kbytes = kXB * kFKP * 4;
    static constexpr int vbytes = 32 * kFVP * 4;
    static constexpr int bytes = kbytes + vbytes;
};

template <int D, int QT>
__global__ void __launch_bounds__(512)
exact_blocked_f32_kernel(const float *__restrict__ q, const float *__restrict__ k,
                         const float *__restrict__ v, float *__restrict__ o, int N, float s2,
                         int wpu)
{
    constexpr int NCT = (D + 15) / 16;
    using X = FBufs;
    extern __shared__ __attribute__((aligned(16))) unsigned char xsm[];
    const int nw = blockDim.x >> 6;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int g = lane >> 4, c = lane & 15;
    const int64_t unit = blockIdx.x / wpu;
    const int wg = int(blockIdx.x - unit * wpu);
    const int64_t base = unit * int64_t(N) * D;
    const float *qu = q + base, *ku = k + base, *vu = v + base;
    float *ou = o + base;
    const int q0 = (wg * nw + w) * 16 * QT;

    if constexpr (16 * NCT > D) {   // V^T rows past D are zero in both buffers
        constexpr int kPad = (16 * NCT - D) * kXB;
        for (int idx = threadIdx.x; idx < 2 * kPad; idx += blockDim.x) {
            const int b = idx / kPad, r = idx % kPad;
            float *vt = reinterpret_cast<float *>(xsm + b * X::bytes + X::kbytes);
            vt[(D + r / kXB) * kFVP + r % kXB] = 0.f;
        }
    }
    // Staging: thread t of the first 256 takes key t / 4, chunk t % 4.
    const bool stager = threadIdx.x < 256;
    const int skey = (threadIdx.x >> 2) & 63, sg = threadIdx.x & 3;
    float kst[8], vst[8];
    auto fetch = [&](int blk) {
        if (stager) {
            const int64_t row = int64_t(blk * kXB + skey) * D + chunk_start<D>(sg);
            load_row8<D>(ku + row, kst);
            load_row8<D>(vu + row, vst);
        }
    };
    auto store = [&](int buf) {
        if (stager) {
            unsigned char *bb = xsm + buf * X::bytes;
            float *krow = reinterpret_cast<float *>(bb) + skey * kFKP + 8 * sg;
            f4 k0, k1;
#pragma unroll
            for (int x = 0; x < 4; ++x) {
                k0[x] = slot_valid<D>(sg, x) ? kst[x] : 0.f;
                k1[x] = slot_valid<D>(sg, 4 + x) ? kst[4 + x] : 0.f;
            }
            reinterpret_cast<f4 *>(krow)[0] = k0;
            reinterpret_cast<f4 *>(krow)[1] = k1;
            float *vt = reinterpret_cast<float *>(bb + X::kbytes);
#pragma unroll
            for (int x = 0; x < 8; ++x)
                if (slot_valid<D>(sg, x))
                    vt[(chunk_start<D>(sg) + x) * kFVP + skey] = vst[x];
        }
    };

    float qf[QT][8];
#pragma unroll
    for (int t = 0; t < QT; ++t)
        load_chunk8<F32, D>(qu + int64_t(q0 + 16 * t + c) * D, g, qf[t]);
    f4 OT[QT][NCT];
    float mref[QT], lsum[QT];
#pragma unroll
    for (int t = 0; t < QT; ++t) {
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
            OT[t][ct] = f4{0.f, 0.f, 0.f, 0.f};
        mref[t] = -INFINITY;
        lsum[t] = 0.f;
    }

    const int nblk = N / kXB;
    fetch(0);
    store(0);
    __syncthreads();
    for (int blk = 0; blk < nblk; ++blk) {
        const int buf = blk & 1;
        if (blk + 1 < nblk)
            fetch(blk + 1);
        const unsigned char *bb = xsm + buf * X::bytes;
        const float *kb = reinterpret_cast<const float *>(bb);
        const float *vt = reinterpret_cast<const float *>(bb + X::kbytes);
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
            float kf[8];   // K row 16kt+c, slots of group g
            {
                const f4 a0 = reinterpret_cast<const f4 *>(kb + (16 * kt + c) * kFKP + 8 * g)[0];
                const f4 a1 = reinterpret_cast<const f4 *>(kb + (16 * kt + c) * kFKP + 8 * g)[1];
#pragma unroll
                for (int x = 0; x < 4; ++x) {
                    kf[x] = a0[x];
                    kf[4 + x] = a1[x];
                }
            }
            f4 vl[NCT];   // V^T tile (ct, kt) as the left operand: lane (g,c) V[16kt+4g+i][16ct+c]
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
                vl[ct] = *reinterpret_cast<const f4 *>(vt + (16 * ct + c) * kFVP + 16 * kt + 4 * g);
#pragma unroll
            for (int t = 0; t < QT; ++t) {
                f4 st = {0.f, 0.f, 0.f, 0.f};   // S^T[key 16kt+4g+i][query q0+16t+c]
#pragma unroll
                for (int x = 0; x < 8; ++x)
                    st = mfma4(kf[x], qf[t][x], st);
                const float lmax = fmaxf(fmaxf(st[0], st[1]), fmaxf(st[2], st[3]));
                if (__builtin_amdgcn_ballot_w64(s2 * lmax > mref[t] + 8.f) != 0) {
                    const float mnew = fmaxf(mref[t], s2 * max_groups(lmax));
                    const float f = fast_exp2(mref[t] - mnew);
                    lsum[t] *= f;
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct)
                        OT[t][ct] *= f;
                    mref[t] = mnew;
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    st[i] = fast_exp2(fmaf(s2, st[i], -mref[t]));
                    lsum[t] += st[i];
                }
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
                    OT[t][ct] = mm16_acc(vl[ct], st, OT[t][ct]);
            }
        }
        if (blk + 1 < nblk)
            store(buf ^ 1);
        __syncthreads();
    }
#pragma unroll
    for (int t = 0; t < QT; ++t) {
        const float inv = __builtin_amdgcn_rcpf(sum_groups(lsum[t]));
        float *orow = ou + int64_t(q0 + 16 * t + c) * D;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int f = 16 * ct + 4 * g + i;
                if (f < D)
                    orow[f] = OT[t][ct][i] * inv;
            }
    }
}

// Query tiles per wave (four from 256 tokens on, so that a K or V fragment
// read from LDS serves four products; one below, so that a workgroup still
// has four waves to stage a block) and waves per workgroup.
constexpr int kXMaxWaves = 8;
inline int exact_qt(int N) { return N >= 256 ? 4 : 1; }

bool exact_blocked_ok(const Problem &p)
{
    if (p.N % kXB != 0 || !tiled_width(p.d) || p.d % 2 != 0)
        return false;
    // bf16: 16-byte row pieces at even elements and paired output stores
    const uintptr_t mis = uintptr_t(p.q) | uintptr_t(p.k) | uintptr_t(p.v) | uintptr_t(p.o);
    if (p.dtype == 1 && mis % 4 != 0)
        return false;
    // whole-wave query groups that divide evenly into workgroups of at least
    // four waves, and the grid under 2^32 work-items
    const int tiles = p.N / (16 * exact_qt(p.N));
    const int nw = tiles < kXMaxWaves ? tiles : kXMaxWaves;
    if (nw < 4 || tiles % nw != 0)
        return false;
    return p.units * int64_t(p.N) * 64 / (16 * exact_qt(p.N)) < (int64_t(1) << 32);
}

template <int D, int QT>
void launch_exact_blocked_qt(const Problem &p, hipStream_t stream)
{
    const int tiles = p.N / (16 * QT);              // wave-sized query groups per unit
    const int nw = tiles < kXMaxWaves ? tiles : kXMaxWaves;
    const int wpu = tiles / nw;
    if (p.dtype == 1) {
        const size_t lds = 2 * size_t(XBufs<D>::bytes);
        hipLaunchKernelGGL((exact_blocked_kernel<D, QT>), dim3(unsigned(p.units * wpu)),
                           dim3(64 * nw), lds, stream, static_cast<const uint16_t *>(p.q),
                           static_cast<const uint16_t *>(p.k), static_cast<const uint16_t *>(p.v),
                           static_cast<uint16_t *>(p.o), p.N, p.scale * kLog2e, wpu);
    } else {
        const size_t lds = 2 * size_t(FBufs::bytes);
        hipLaunchKernelGGL((exact_blocked_f32_kernel<D, QT>), dim3(unsigned(p.units * wpu)),
                           dim3(64 * nw), lds, stream, static_cast<const float *>(p.q),
                           static_cast<const float *>(p.k), static_cast<const float *>(p.v),
                           static_cast<float *>(p.o), p.N, p.scale * kLog2e, wpu);
    }
}

template <int D>
void launch_exact_blocked(const Problem &p, hipStream_t stream)
{
    if (exact_qt(p.N) == 4)
        launch_exact_blocked_qt<D, 4>(p, stream);
    else
        launch_exact_blocked_qt<D, 1>(p, stream);
}

void launch_exact_blocked_d(const Problem &p, hipStream_t stream)
{
    switch (p.d) {
    case 8: launch_exact_blocked<8>(p, stream); break;
    case 12: launch_exact_blocked<12>(p, stream); break;
    case 16: launch_exact_blocked<16>(p, stream); break;
    case 20: launch_exact_blocked<20>(p, stream); break;
    case 24: launch_exact_blocked<24>(p, stream); break;
    case 28: launch_exact_blocked<28>(p, stream); break;
    case 30: launch_exact_blocked<30>(p, stream); break;
    default: launch_exact_blocked<32>(p, stream); break;
    }
}

// V^T of one unit in LDS for the bf16 path; larger windows run the fp32
// matrix cores on the (exactly converted) bf16 inputs instead.
constexpr size_t kExactLdsMax = 128 * 1024;

template <class E, int D>
void launch_exact_tiled(const Problem &p, hipStream_t stream)
{
    const int NT = p.N / 16;
    const int qblocks = (NT + kExactWaves - 1) / kExactWaves;
    const size_t lds = size_t(32) * (p.N + 8) * 2;
    const auto *q = static_cast<const typename E::T *>(p.q);
    const auto *k = static_cast<const typename E::T *>(p.k);
    const auto *v = static_cast<const typename E::T *>(p.v);
    auto *o = static_cast<typename E::T *>(p.o);
    const dim3 grid(unsigned(p.units * qblocks)), block(64 * kExactWaves);
    if (E::bytes == 2 && lds <= kExactLdsMax)
        hipLaunchKernelGGL((exact_tiled_kernel<E, D, true>), grid, block, lds, stream, q, k, v,
                           o, p.N, p.scale * kLog2e, qblocks);
    else
        hipLaunchKernelGGL((exact_tiled_kernel<E, D, false>), grid, block, 0, stream, q, k, v,
                           o, p.N, p.scale * kLog2e, qblocks);
}

template <class E>
void launch_exact_tiled_e(const Problem &p, hipStream_t stream)
{
    switch (p.d) {
    case 8: launch_exact_tiled<E, 8>(p, stream); break;
    case 12: launch_exact_tiled<E, 12>(p, stream); break;
    case 16: launch_exact_tiled<E, 16>(p, stream); break;
    case 20: launch_exact_tiled<E, 20>(p, stream); break;
    case 24: launch_exact_tiled<E, 24>(p, stream); break;
    case 28: launch_exact_tiled<E, 28>(p, stream); break;
    case 30: launch_exact_tiled<E, 30>(p, stream); break;
    default: launch_exact_tiled<E, 32>(p, stream); break;
    }
}

bool exact_tiled_ok(const Problem &p)
{
    if (p.N % 32 != 0 || !tiled_width(p.d))
        return false;
    // fewer than 2^32 work-items in the grid; otherwise the rows kernel runs
    if (p.units * int64_t((p.N / 16 + kExactWaves - 1) / kExactWaves) * 64 * kExactWaves >=
        (int64_t(1) << 32))
        return false;
    if (p.dtype == 1) {
        const uintptr_t mis = uintptr_t(p.q) | uintptr_t(p.k) | uintptr_t(p.v);
        if (mis % 4 != 0)
            return false;
    }
    return true;
}

template <class E>
hipError_t launch_exact_t(const Problem &p, hipStream_t stream)
{
    if (exact_blocked_ok(p)) {
        launch_exact_blocked_d(p, stream);
        return hipGetLastError();
    }
    if (exact_tiled_ok(p)) {
        launch_exact_tiled_e<E>(p, stream);
        return hipGetLastError();
    }
    const dim3 grid(unsigned(p.units), unsigned((p.N + kThreads - 1) / kThreads));
    const auto *q = static_cast<const typename E::T *>(p.q);
    const auto *k = static_cast<const typename E::T *>(p.k);
    const auto *v = static_cast<const typename E::T *>(p.v);
    auto *o = static_cast<typename E::T *>(p.o);
    if (p.d <= 64)
        hipLaunchKernelGGL((exact_rows_kernel<E, 64>), grid, dim3(kThreads), 0, stream, q, k, v,
                           o, p.N, p.d, p.scale);
    else
        hipLaunchKernelGGL((exact_rows_kernel<E, 128>), grid, dim3(kThreads), 0, stream, q, k,
                           v, o, p.N, p.d, p.scale);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_exact(const Problem &p, hipStream_t stream)
{
    return p.dtype == 0 ? launch_exact_t<F32>(p, stream) : launch_exact_t<BF16>(p, stream);
}

}  // namespace nystra
