// MFMA-tiled PnP-Nystra kernel for large windows (N a multiple of 16, e.g.
// 16x16 and 32x32 windows; m <= 64 landmarks; d_h in {8, 16, 24, 30, 32}).
//
// One workgroup computes one (window, head) unit with MT = ceil(m / 16)
// wavefronts; wave w owns landmark tile w (landmarks 16w .. 16w+15):
//   1. Step 1: each lane averages the patch of its own landmark straight from
//      global memory (any pooling grid), producing Qbar rows in registers and
//      Kbar rows in LDS.
//   2. Step 3, G_U side: the wave streams all N keys twice -- once for the row
//      maxima m_U of its landmarks, once for G_U^n and T = G_U^n [V | 1].
//   3. Step 2 and Step 4: the wave builds its row tile of A = G_A^n; the m x m
//      pseudo-inverse iteration runs with each wave computing its row tile of
//      every product, the right-hand operands exchanged through LDS.
//   4. Steps 5-6: W = Z T, exchanged through LDS.
//   5. Steps 3 (G_L side), 6 and 7: the waves split the token tiles; per tile
//      S_L, the row max over all landmarks, G_L^n, O = G_L^n W, O_D, divide.
// Every contraction runs on v_mfma_f32_16x16x4f32 with the register tiles of
// tile_common.hpp.  Matrices shared between waves sit in LDS row-major with a
// padded pitch: a right-hand operand tile is read as four strided words per
// lane, the transpose of an own-row tile as one 16-byte word per lane.
#include "internal.hpp"
#include "tile_common.hpp"

namespace nystra {
namespace {

using namespace tile;

constexpr int kTS = 36;   // pitch of [landmark][feature] tables (Kbar, T, W)

struct LargeArgs {
    int64_t units;
    int N, m, iters;
    float s2;          // logit scale in base-2 units (scale * log2 e)
    float inv_patch;   // 1 / tokens per pooling patch
    int cols, pr, pc, gc;   // pooling grid
};

// LDS carve-up (floats) for MT landmark tiles.
template <int MT>
struct LargeLds {
    static constexpr int M = 16 * MT;
    static constexpr int P = M + 4;   // pitch of the m x m matrices
    static constexpr int kbar = 0;
    static constexpr int colpart = kbar + M * kTS;      // [MT][M] column-sum partials
    static constexpr int rowmax = colpart + MT * M;     // [MT] row-sum maxima (padded)
    static constexpr int zb = rowmax + 4;
    static constexpr int ya = zb + M * P;
    static constexpr int yb = ya + M * P;               // also the own-row X scratch
    static constexpr int vec = yb + M * P;              // [MT][64]
    static constexpr int tab_len = M * kTS + M;         // table + its denominator column
    static constexpr bool tab_in_y = tab_len <= M * P;  // T in ya, W in yb after the iteration
    static constexpr int tb = tab_in_y ? ya : vec + MT * 64;
    static constexpr int wb = tab_in_y ? yb : tb + tab_len;
    static constexpr int total = tab_in_y ? vec + MT * 64 : wb + tab_len;
};

// Right-hand operand (D-layout) of tile (a, b) of a row-major LDS matrix.
template <int P>
__device__ inline f4 read_r(const float *B, int a, int b, int g, int c)
{
    f4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i)
        r[i] = B[(16 * a + 4 * g + i) * P + 16 * b + c];
    return r;
}

// Transposed tile (a, b) in D-layout: lane (g, c) gets B[16a + c][16b + 4g + i].
template <int P>
__device__ inline f4 read_lt(const float *B, int a, int b, int g, int c)
{
    return *reinterpret_cast<const f4 *>(B + (16 * a + c) * P + 16 * b + 4 * g);
}

// Stores a D-layout tile as tile (a, b) of a row-major LDS matrix.
template <int P>
__device__ inline void write_tile(float *B, int a, int b, f4 v, int g, int c)
{
#pragma unroll
    for (int i = 0; i < 4; ++i)
        B[(16 * a + 4 * g + i) * P + 16 * b + c] = v[i];
}

template <class E, int MT, int D>
__global__ void __launch_bounds__(64 * MT)
tiled_large_kernel(const typename E::T *__restrict__ q, const typename E::T *__restrict__ k,
                   const typename E::T *__restrict__ v, typename E::T *__restrict__ o,
                   LargeArgs a)
{
    using L = LargeLds<MT>;
    constexpr int M = L::M, P = L::P, d = D;
    extern __shared__ float lds[];
    float *kbar = lds + L::kbar, *colpart = lds + L::colpart;
    float *rowmax = lds + L::rowmax, *Zb = lds + L::zb, *Ya = lds + L::ya, *Yb = lds + L::yb;
    float *Tb = lds + L::tb, *Wb = lds + L::wb;

    const int lt = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int g = lane >> 4, c = lane & 15;
    float *vec = lds + L::vec + 64 * lt;
    const int m = a.m, N = a.N, NT = a.N >> 4;
    const int l = 16 * lt + c;            // this lane's landmark
    const bool lval = l < m;
    const int64_t base = int64_t(blockIdx.x) * N * d;
    const typename E::T *qu = q + base, *ku = k + base, *vu = v + base;
    typename E::T *ou = o + base;

    // ---- Step 1: means of this landmark's patch (rows r0.., cols c0..).
    float qb[8], kbv[8];
#pragma unroll
    for (int s = 0; s < 8; ++s)
        qb[s] = kbv[s] = 0.f;
    {
        const int le = lval ? l : m - 1;   // padding lanes read a valid patch, then drop it
        const int r0 = (le / a.gc) * a.pr, c0 = (le % a.gc) * a.pc;
        for (int r = r0; r < r0 + a.pr; ++r)
            for (int cc = c0; cc < c0 + a.pc; ++cc) {
                float x[8], y[8];
                const int64_t t = int64_t(r) * a.cols + cc;
                load_chunk8<E, D>(qu + t * d, g, x);
                load_chunk8<E, D>(ku + t * d, g, y);
#pragma unroll
                for (int s = 0; s < 8; ++s) {
                    qb[s] += x[s];
                    kbv[s] += y[s];
                }
            }
        const float sc = lval ? a.inv_patch : 0.f;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            qb[s] *= sc;
            kbv[s] *= sc;
        }
    }
#pragma unroll
    for (int s = 0; s < 8; ++s)
        if (slot_valid<D>(g, s))
            kbar[l * kTS + chunk_start<D>(g) + s] = kbv[s];

    // ---- Step 3, G_U side, pass 1: m_U of this landmark over all N keys.
    float mx = -INFINITY;
    {
        float kn[8];
        load_chunk8<E, D>(ku + int64_t(c) * d, g, kn);
        for (int tt = 0; tt < NT; ++tt) {
            float kr[8];
#pragma unroll
            for (int s = 0; s < 8; ++s)
                kr[s] = kn[s];
            load_chunk8<E, D>(ku + int64_t(16 * min(tt + 1, NT - 1) + c) * d, g, kn);
            f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < 8; ++s)
                acc = mfma4(kr[s], qb[s], acc);
            mx = fmaxf(mx, fmaxf(fmaxf(acc[0], acc[1]), fmaxf(acc[2], acc[3])));
        }
    }
    const float mu = a.s2 * max_groups(mx);   // m_U of landmark l (base-2 units)

    // ---- pass 2: G_U^n and T = G_U^n V, T_D = G_U^n 1.
    // T[ct] lane (g,c): T[landmark 16lt+4g+i][feature 16ct+c].
    f4 T[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
    float tden = 0.f;
    {
        float kn[8], vn[2][4];
        auto load_tile = [&](int tt, float *kx, float (*vx)[4]) {
            load_chunk8<E, D>(ku + int64_t(16 * tt + c) * d, g, kx);
#pragma unroll
            for (int ct = 0; ct < 2; ++ct) {
                const int f = 16 * ct + c;
#pragma unroll
                for (int s = 0; s < 4; ++s) {
                    const float x = E::load(vu, int64_t(16 * tt + 4 * g + s) * d + min(f, d - 1));
                    vx[ct][s] = f < d ? x : 0.f;
                }
            }
        };
        load_tile(0, kn, vn);
        for (int tt = 0; tt < NT; ++tt) {
            float kr[8], vr[2][4];
#pragma unroll
            for (int s = 0; s < 8; ++s)
                kr[s] = kn[s];
#pragma unroll
            for (int ct = 0; ct < 2; ++ct)
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    vr[ct][s] = vn[ct][s];
            load_tile(min(tt + 1, NT - 1), kn, vn);
            f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < 8; ++s)
                acc = mfma4(kr[s], qb[s], acc);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                acc[i] = lval ? fast_exp2(fmaf(a.s2, acc[i], -mu)) : 0.f;
                tden += acc[i];
            }
#pragma unroll
            for (int ct = 0; ct < 2; ++ct)
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    T[ct] = mfma4(acc[s], vr[ct][s], T[ct]);
        }
    }
    tden = sum_groups(tden);   // T_D of landmark l
    __syncthreads();           // Kbar complete

    // ---- Step 2: this wave's row tile of A = G_A^n, in transposed form:
    // ALT[j] lane (g,c): A[16lt + c][16j + 4g + i].
    f4 ALT[MT];
#pragma unroll
    for (int j = 0; j < MT; ++j) {
        f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            const float kv = slot_valid<D>(g, s)
                                 ? kbar[(16 * j + c) * kTS + chunk_start<D>(g) + s] : 0.f;
            acc = mfma4(kv, qb[s], acc);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
            ALT[j][i] = (lval && 16 * j + 4 * g + i < m) ? fast_exp2(fmaf(a.s2, acc[i], -mu))
                                                         : 0.f;
    }

    // ---- Step 4: Z_0 = A^T / (||A||_1 ||A||_inf).
    {
        float rs = 0.f;
#pragma unroll
        for (int j = 0; j < MT; ++j)
            rs += ALT[j][0] + ALT[j][1] + ALT[j][2] + ALT[j][3];
        rs = sum_groups(rs);                        // sum of row l
        const float rmax = max_groups(max_row(rs));
        if (lane == 0)
            rowmax[lt] = rmax;
#pragma unroll
        for (int j = 0; j < MT; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float cs = sum_row(ALT[j][i]);   // column 16j+4g+i over this tile's rows
                if (c == 0)
                    colpart[lt * M + 16 * j + 4 * g + i] = cs;
            }
    }
    __syncthreads();
    float alpha;
    {
        float cs = 0.f;
        if (lane < M)
            for (int w = 0; w < MT; ++w)
                cs += colpart[w * M + lane];
        const float n1 = max_groups(max_row(cs));
        float ninf = 0.f;
        for (int w = 0; w < MT; ++w)
            ninf = fmaxf(ninf, rowmax[w]);
        alpha = 1.0f / (n1 * ninf);
    }
    // Z_0[j][lt] = alpha (A[lt][j])^T, whose D-layout is alpha * ALT[j].
#pragma unroll
    for (int j = 0; j < MT; ++j)
        write_tile<P>(Zb, j, lt, ALT[j] * alpha, g, c);
    __syncthreads();
    f4 ZLT[MT];   // ZLT[j] lane (g,c): Z[16lt + c][16j + 4g + i]
#pragma unroll
    for (int j = 0; j < MT; ++j)
        ZLT[j] = read_lt<P>(Zb, lt, j, g, c);
    f4 eye;   // identity of the m x m block on this wave's diagonal tile
#pragma unroll
    for (int i = 0; i < 4; ++i)
        eye[i] = (4 * g + i == c && lval) ? 1.f : 0.f;

    // Iteration: X = A Z; Z <- Z (13I - X (15I - X (7I - X))) / 4, each wave
    // producing its row tile of every product.
    for (int it = 0; it < a.iters; ++it) {
        f4 X[MT];
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < MT; ++kk) {
                const f4 zr = read_r<P>(Zb, kk, j, g, c);
                acc = mfma4(ALT[kk][0], zr[0], acc);
                acc = mfma4(ALT[kk][1], zr[1], acc);
                acc = mfma4(ALT[kk][2], zr[2], acc);
                acc = mfma4(ALT[kk][3], zr[3], acc);
            }
            X[j] = acc;
        }
        // own-row transpose of X through Yb (free at this point)
#pragma unroll
        for (int j = 0; j < MT; ++j)
            write_tile<P>(Yb, lt, j, X[j], g, c);
        wave_sync();
        f4 XLT[MT];
#pragma unroll
        for (int j = 0; j < MT; ++j)
            XLT[j] = read_lt<P>(Yb, lt, j, g, c);
#pragma unroll
        for (int j = 0; j < MT; ++j)
            write_tile<P>(Ya, lt, j, (j == lt ? eye * 7.f : f4{0.f, 0.f, 0.f, 0.f}) - X[j], g, c);
        __syncthreads();
        f4 Y[MT];
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < MT; ++kk)
                acc += mm16(XLT[kk], read_r<P>(Ya, kk, j, g, c));
            Y[j] = (j == lt ? eye * 15.f : f4{0.f, 0.f, 0.f, 0.f}) - acc;
        }
#pragma unroll
        for (int j = 0; j < MT; ++j)
            write_tile<P>(Yb, lt, j, Y[j], g, c);
        __syncthreads();
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < MT; ++kk)
                acc += mm16(XLT[kk], read_r<P>(Yb, kk, j, g, c));
            Y[j] = (j == lt ? eye * 13.f : f4{0.f, 0.f, 0.f, 0.f}) - acc;
        }
#pragma unroll
        for (int j = 0; j < MT; ++j)
            write_tile<P>(Ya, lt, j, Y[j], g, c);
        __syncthreads();
        f4 Zn[MT];
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < MT; ++kk)
                acc += mm16(ZLT[kk], read_r<P>(Ya, kk, j, g, c));
            Zn[j] = acc * 0.25f;
        }
#pragma unroll
        for (int j = 0; j < MT; ++j)
            write_tile<P>(Zb, lt, j, Zn[j], g, c);
        wave_sync();
#pragma unroll
        for (int j = 0; j < MT; ++j)
            ZLT[j] = read_lt<P>(Zb, lt, j, g, c);
        __syncthreads();
    }

    // ---- Steps 5-6 re-associated: W = Z T and W_D = Z T_D.
    constexpr int TDo = M * kTS;   // offset of the denominator column in a table
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
        write_tile<kTS>(Tb, lt, ct, T[ct], g, c);
    if (g == 0)
        Tb[TDo + l] = tden;
    __syncthreads();
    f4 Wt[2];
#pragma unroll
    for (int ct = 0; ct < 2; ++ct) {
        f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < MT; ++kk)
            acc += mm16(ZLT[kk], read_r<kTS>(Tb, kk, ct, g, c));
        Wt[ct] = acc;
    }
    float wden = 0.f;
#pragma unroll
    for (int kk = 0; kk < MT; ++kk) {
        const f4 td = *reinterpret_cast<const f4 *>(Tb + TDo + 16 * kk + 4 * g);
        wden += ZLT[kk][0] * td[0] + ZLT[kk][1] * td[1] + ZLT[kk][2] * td[2] +
                ZLT[kk][3] * td[3];
    }
    wden = sum_groups(wden);
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
        write_tile<kTS>(Wb, lt, ct, Wt[ct], g, c);
    if (g == 0)
        Wb[TDo + l] = wden;
    __syncthreads();

    // ---- Steps 3 (G_L side), 6 and 7 over this wave's token tiles.
    f4 WR[MT][2], wdv[MT];
    float kb[MT][8];
#pragma unroll
    for (int kk = 0; kk < MT; ++kk) {
        WR[kk][0] = read_r<kTS>(Wb, kk, 0, g, c);
        WR[kk][1] = read_r<kTS>(Wb, kk, 1, g, c);
        wdv[kk] = *reinterpret_cast<const f4 *>(Wb + TDo + 16 * kk + 4 * g);
#pragma unroll
        for (int s = 0; s < 8; ++s)
            kb[kk][s] = slot_valid<D>(g, s)
                            ? kbar[(16 * kk + c) * kTS + chunk_start<D>(g) + s] : 0.f;
    }
    float qn[8];
    load_chunk8<E, D>(qu + int64_t(16 * min(lt, NT - 1) + c) * d, g, qn);
    for (int tt = lt; tt < NT; tt += MT) {
        float qr[8];
#pragma unroll
        for (int s = 0; s < 8; ++s)
            qr[s] = qn[s];
        load_chunk8<E, D>(qu + int64_t(16 * min(tt + MT, NT - 1) + c) * d, g, qn);
        f4 glT[MT];   // lane (g,c): G_L^n[token 16tt+c][landmark 16kk+4g+i]
        float ml = -INFINITY;
#pragma unroll
        for (int kk = 0; kk < MT; ++kk) {
            f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < 8; ++s)
                acc = mfma4(kb[kk][s], qr[s], acc);
            glT[kk] = acc;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (16 * kk + 4 * g + i < m)
                    ml = fmaxf(ml, acc[i]);
        }
        ml = a.s2 * max_groups(ml);
        float od = 0.f;
#pragma unroll
        for (int kk = 0; kk < MT; ++kk)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float e = (16 * kk + 4 * g + i < m) ? fast_exp2(fmaf(a.s2, glT[kk][i], -ml))
                                                          : 0.f;
                glT[kk][i] = e;
                od = fmaf(e, wdv[kk][i], od);
            }
        od = sum_groups(od);
        const f4 odr = by_rows(od, vec, g, c);   // O_D[16tt + 4g + i]
        f4 rcp;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            rcp[i] = __builtin_amdgcn_rcpf(odr[i]);
#pragma unroll
        for (int ct = 0; ct < 2; ++ct) {
            f4 on = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < MT; ++kk)
                on += mm16(glT[kk], WR[kk][ct]);
            const int f = 16 * ct + c;
            if (f < d) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    E::store(ou, int64_t(16 * tt + 4 * g + i) * d + f, on[i] * rcp[i]);
            }
        }
    }
}

template <class E, int MT, int D>
void launch_large(const Problem &p, const LargeArgs &a, hipStream_t stream)
{
    const size_t lds = size_t(LargeLds<MT>::total) * sizeof(float);
    hipLaunchKernelGGL((tiled_large_kernel<E, MT, D>), dim3(unsigned(p.units)), dim3(64 * MT),
                       lds, stream, static_cast<const typename E::T *>(p.q),
                       static_cast<const typename E::T *>(p.k),
                       static_cast<const typename E::T *>(p.v),
                       static_cast<typename E::T *>(p.o), a);
}

template <class E, int D>
void launch_large_m(const Problem &p, const LargeArgs &a, hipStream_t stream)
{
    switch ((p.m + 15) / 16) {
    case 1: launch_large<E, 1, D>(p, a, stream); break;
    case 2: launch_large<E, 2, D>(p, a, stream); break;
    case 3: launch_large<E, 3, D>(p, a, stream); break;
    default: launch_large<E, 4, D>(p, a, stream); break;
    }
}

template <class E>
void launch_large_e(const Problem &p, const LargeArgs &a, hipStream_t stream)
{
    switch (p.d) {
    case 8: launch_large_m<E, 8>(p, a, stream); break;
    case 16: launch_large_m<E, 16>(p, a, stream); break;
    case 24: launch_large_m<E, 24>(p, a, stream); break;
    case 30: launch_large_m<E, 30>(p, a, stream); break;
    default: launch_large_m<E, 32>(p, a, stream); break;
    }
}

}  // namespace

bool tiled_large_supported(const Problem &p)
{
    if (p.N % 16 != 0 || p.m > 64 || !tiled_width(p.d))
        return false;
    if (p.dtype == 1) {   // 16-byte row pieces of bf16 need 4-byte aligned rows
        const uintptr_t mis = uintptr_t(p.q) | uintptr_t(p.k) | uintptr_t(p.v);
        if (mis % 4 != 0)
            return false;
    }
    return true;
}

hipError_t launch_tiled_large(const Problem &p, hipStream_t stream)
{
    LargeArgs a;
    a.units = p.units;
    a.N = p.N;
    a.m = p.m;
    a.iters = p.iters;
    a.s2 = p.scale * kLog2e;
    a.inv_patch = 1.0f / float(p.geo.pr * p.geo.pc);
    a.cols = p.geo.cols;
    a.pr = p.geo.pr;
    a.pc = p.geo.pc;
    a.gc = p.geo.gc;
    if (p.dtype == 0)
        launch_large_e<F32>(p, a, stream);
    else
        launch_large_e<BF16>(p, a, stream);
    return hipGetLastError();
}

}  // namespace nystra
