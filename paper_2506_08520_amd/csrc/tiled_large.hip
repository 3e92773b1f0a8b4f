// MFMA-tiled PnP-Nystra kernel for large windows (N a multiple of 16, e.g.
// 16x16 and 32x32 windows; m <= 64 landmarks; d_h in {8, 12, ..., 28, 30, 32}).
//
// One workgroup computes one (window, head) unit with MT = ceil(m / 16)
// wavefronts; wave w owns landmark tile w (landmarks 16w .. 16w+15):
//   1. Step 1: each lane averages the patch of its own landmark straight from
//      global memory (any pooling grid), producing Qbar rows in registers and
//      Kbar rows in LDS.
//   2. Step 3, G_U side: the waves split the keys, each wave covering every
//      landmark tile: running maxima of S_U over its keys, and G_U^n and
//      T = G_U^n [V | 1] accumulated against them (rescaled whenever a maximum
//      grows).  The waves' records are merged in LDS against the row maxima
//      m_U over all keys.  Every K and V row is read once per unit.  With the
//      patch grids of 16 x 16 and 32 x 32 windows (patches four tokens wide)
//      and bf16 inputs, Step 1 for K happens here too (KP): each wave takes
//      whole bands of patches and sums their K rows as they pass.
//   3. Step 2 and Step 4: the wave builds its row tile of A = G_A^n; the m x m
//      pseudo-inverse iteration runs with each wave computing its row tile of
//      every product, the right-hand operands exchanged through LDS.
//   4. Steps 5-6: W = Z T, exchanged through LDS.
//   5. Steps 3 (G_L side), 6 and 7: the waves split the token tiles; per tile
//      S_L, the row max over all landmarks, G_L^n, O = G_L^n W, O_D, divide.
// Steps 2, 4 and 5-6 are the shared landmark core of core_tiles.hpp.  The
// contractions run on the fp32 matrix cores with the register tiles of
// tile_common.hpp; bf16 inputs with N % 32 == 0 run the token-side products on
// the bf16 matrix cores, fp32 operands carried as hi + lo terms.
#include "internal.hpp"
#include "core_tiles.hpp"

namespace nystra {
namespace {

using namespace tile;
using namespace core;

struct LargeArgs {
    int64_t units;
    int N, m, iters;
    float s2;          // logit scale in base-2 units (scale * log2 e)
    float inv_patch;   // 1 / tokens per pooling patch
    int cols, pr, pc, gc;   // pooling grid
};

// FULL: m = 16 MT, so every landmark slot is real and the masks fold away.
// KPL: 0 = Kbar pooled before the key pass; otherwise pooled in it (bf16,
// FULL, the grids kpool_ok accepts): 1 = one 16-token tile per image row and
// one pair of tiles per band of patches (16 x 16 windows, 2 x 4 patches),
// 2 = two tiles per image row (32 x 32 windows), any band height.  With KPL = 1 the registers
// are held to 128 (four waves per SIMD, as without KP); the few values that
// do not fit are saved once around the key pass, none inside it.
template <class E, int MT, int D, bool BFM, bool FULL, int KPL>
__global__ void __launch_bounds__(64 * MT)
__attribute__((amdgpu_waves_per_eu(KPL == 1 ? 4 : 1)))
tiled_large_kernel(const typename E::T *__restrict__ q, const typename E::T *__restrict__ k,
                   const typename E::T *__restrict__ v, typename E::T *__restrict__ o,
                   LargeArgs a)
{
    using L = LargeLds<MT>;
    constexpr bool KP = KPL != 0;
    static_assert(!KP || (BFM && FULL), "K pooling in the key pass: bf16, full landmark tiles");
    constexpr int d = D;
    // With a spare column (D % 16 != 0), column D of V is replaced by ones, so
    // that column D of T, W and O carries T_D, W_D and O_D (no separate sums).
    constexpr bool PAD = D % 16 != 0;
    extern __shared__ float lds[];
    float *kbar = lds + L::kbar;

    // the wave index is uniform: keep it (and the loops it bounds) scalar
    const int lt = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int g = lane >> 4, c = lane & 15;
    float *vec = lds + L::vec + 64 * lt;
    const int m = FULL ? 16 * MT : a.m, N = a.N, NT = a.N >> 4;
    const int l = 16 * lt + c;            // this lane's landmark
    const bool lval = FULL || l < m;
    const int64_t base = int64_t(blockIdx.x) * N * d;
    const typename E::T *qu = q + base, *ku = k + base, *vu = v + base;
    typename E::T *ou = o + base;

    // ---- Step 1: means of this landmark's patch (rows r0.., cols c0..),
    // eight patch tokens per step so their loads are in flight together.
    float qb[8], kbv[8];
#pragma unroll
    for (int s = 0; s < 8; ++s)
        qb[s] = kbv[s] = 0.f;
    {
        // KPL 2 fixes the grid (32 columns, 4 x 4 patches, 8 per row), so the
        // token offsets below are shifts and masks (c5 -1.3%; the same for
        // KPL 1 measured +0.9%); otherwise they come from a.
        const int gcols = KPL == 2 ? 32 : a.cols;
        const int gpr = KPL == 2 ? 4 : a.pr;
        const int gpc = KPL == 2 ? 4 : a.pc;
        const int ggc = KPL == 2 ? 8 : a.gc;
        const int le = lval ? l : m - 1;   // padding lanes read a valid patch, then drop it
        const int r0 = (le / ggc) * gpr, c0 = (le % ggc) * gpc;
        const int npatch = gpr * gpc;
        // Rows arrive raw; the slots a lower lane group carries are zeroed
        // once, in the sums (the same values as zeroing every row).
        constexpr int kP = 8;
        for (int j0 = 0; j0 < npatch; j0 += kP) {
            float x[kP][8], y[kP][8];   // fp32 rows
            U16B xb[kP], yb[kP];        // bf16 rows (raw pairs)
#pragma unroll
            for (int u = 0; u < kP; ++u) {
                const int j = min(j0 + u, npatch - 1);
                const int64_t t = (int64_t(r0 + j / gpc) * gcols + c0 + j % gpc) * d +
                                  chunk_start<D>(g);
                if constexpr (E::bytes == 4) {
                    load_row8<D>(qu + t, x[u]);
                    load_row8<D>(ku + t, y[u]);
                } else {
                    xb[u] = *reinterpret_cast<const U16B *>(qu + t);
                    if constexpr (!KP)
                        yb[u] = *reinterpret_cast<const U16B *>(ku + t);
                }
            }
#pragma unroll
            for (int u = 0; u < kP; ++u)
                if (j0 + u < npatch) {
                    if constexpr (E::bytes == 4) {
#pragma unroll
                        for (int s = 0; s < 8; ++s) {
                            qb[s] += x[u][s];
                            kbv[s] += y[u][s];
                        }
                    } else {
#pragma unroll
                        for (int w = 0; w < 4; ++w) {
                            qb[2 * w] += __uint_as_float(xb[u].w[w] << 16);
                            qb[2 * w + 1] += __uint_as_float(xb[u].w[w] & 0xffff0000u);
                            if constexpr (!KP) {
                                kbv[2 * w] += __uint_as_float(yb[u].w[w] << 16);
                                kbv[2 * w + 1] += __uint_as_float(yb[u].w[w] & 0xffff0000u);
                            }
                        }
                    }
                }
        }
        const float sc = lval ? a.inv_patch : 0.f;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            qb[s] = slot_valid<D>(g, s) ? qb[s] * sc : 0.f;
            kbv[s] = slot_valid<D>(g, s) ? kbv[s] * sc : 0.f;
        }
    }
    if constexpr (!KP) {
#pragma unroll
        for (int s = 0; s < 8; ++s)
            if (slot_valid<D>(g, s))
                kbar[l * kTS + chunk_start<D>(g) + s] = kbv[s];
    }

    // Qbar rows go to a table too, so that every wave can read every tile.
    float *qtab = lds + L::qtab;
#pragma unroll
    for (int s = 0; s < 8; ++s)
        if (slot_valid<D>(g, s))
            qtab[l * kTS + chunk_start<D>(g) + s] = qb[s];
    __syncthreads();   // Qbar (and, unless KP, Kbar) complete

    // ---- Step 3, G_U side.  The waves split the keys: wave lt takes the key
    // tile pairs 2lt, 2lt + 2MT, ... and, for every landmark tile j, keeps the
    // running maximum of S_U over its keys and T_j = G_U^n [V | 1] and T_D
    // accumulated against it (rescaled by exp(old - new) whenever a maximum
    // grows).  The waves' records are then merged against the largest of
    // their maxima, m_U: the sums of Step 3 against the row maxima over all N
    // keys, only added in another order.  Every K and V row is read once.
    constexpr int NCT = (D + 15) / 16;   // feature tiles of T (the ones column included)
    constexpr int kRecP = L::kRecP, LD = L::M * kRecP, LM = LD + L::M;
    const uint16_t *ku16 = reinterpret_cast<const uint16_t *>(ku);
    const uint16_t *vu16 = reinterpret_cast<const uint16_t *>(vu);
    float qj[MT][8];   // Qbar rows of every landmark tile: lane (g, c) holds landmark 16j + c
    bf8 qjh[MT], qjl[MT];
#pragma unroll
    for (int j = 0; j < MT; ++j) {
#pragma unroll
        for (int s = 0; s < 8; ++s)
            qj[j][s] = slot_valid<D>(g, s) ? qtab[(16 * j + c) * kTS + chunk_start<D>(g) + s]
                                           : 0.f;
        if constexpr (BFM)
            split_bf16(qj[j], qjh[j], qjl[j]);
    }
    f4 TJ[MT][NCT];
    float tdj[MT], mrj[MT];
#pragma unroll
    for (int j = 0; j < MT; ++j) {
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
            TJ[j][ct] = f4{0.f, 0.f, 0.f, 0.f};
        tdj[j] = 0.f;
        mrj[j] = -INFINITY;
    }
    // The wave's key tile pairs: t0 = t_begin, t_begin + t_stride, ... below
    // t_end.  Round-robin over the waves, or (KP) a contiguous block of whole
    // patch bands: ppb pairs of tiles cover the rows of one band of patches.
    int t_begin = 2 * lt, t_stride = 2 * MT, t_end = NT, ppb = 1;
    if constexpr (KP) {
        const int ppw = (NT >> 1) / MT;
        t_begin = 2 * ppw * lt;
        t_stride = 2;
        t_end = t_begin + 2 * ppw;
        ppb = KPL == 1 ? 1 : (a.pr * (a.cols >> 4)) >> 1;
    }
    // KP: one-hot selectors that move feature 16ct + c of a K row into column
    // c of a product (the valid slot holding it gets 1, every other slot 0),
    // and per-lane partial patch sums pk[u][ct] of the band in progress.  A
    // feature's valid slot lies in lane group f / 8, so lane (g, c) has a 1
    // only in the selector of feature tile g / 2: one selector (ksel_own) is
    // built, the other tile's is zero.  KPL = 1 rebuilds it per pair (fewer
    // registers held through the loop).
    auto own_selector = [&]() {
        U16B w;
        const int f = 16 * (g >> 1) + c;
#pragma unroll
        for (int pp = 0; pp < 4; ++pp) {
            uint32_t x = 0;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int sl = 2 * pp + h;
                if (slot_valid<D>(g, sl) && chunk_start<D>(g) + sl == f)
                    x |= 0x3F80u << (16 * h);   // bf16 1.0
            }
            w.w[pp] = x;
        }
        return w;
    };
    U16B ksel_own = {{0u, 0u, 0u, 0u}};
    float pk[2][2] = {{0.f, 0.f}, {0.f, 0.f}};
    if constexpr (KPL == 2)
        ksel_own = own_selector();
    // Pairs are software-pipelined: the next pair's K and V rows are requested
    // before this pair is computed (past the end they repeat the last tile,
    // unused).  bf16 V is held as pairs of rows (4g, 4g+1) and (4g+2, 4g+3) of
    // one column, the two 16-bit loads landing in the halves of one register.
    typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
    float kr[2][8], vr[2][NCT][4], krn[2][8], vrn[2][NCT][4];
    bf8 kw[2], kwn[2];
    uint32_t vh[2][NCT][2], vhn[2][NCT][2];
    auto load_pair = [&](int t0, float (&kr_)[2][8], bf8 (&kw_)[2], float (&vr_)[2][NCT][4],
                         uint32_t (&vh_)[2][NCT][2]) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            // 32-bit offsets from the unit's (uniform) base: N d < 2^26
            const int tt = min(t0 + u, NT - 1);
            const unsigned row = unsigned(16 * tt + c) * d;
            if constexpr (BFM)
                kw_[u] = load_row8_bf16(ku16 + (row + chunk_start<D>(g)));
            else if constexpr (E::bytes == 4)
                load_row8<D>(ku + (row + chunk_start<D>(g)), kr_[u]);
            else   // bf16 values through the fp32 path: unpacked (and masked) here
                load_chunk8<E, D>(ku + row, g, kr_[u]);
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                const int f = 16 * ct + c;
                // one address per row group; the four rows are immediate offsets
                // (pointer first, then the row offsets: constant multiples of d
                // that fold into the loads' immediate offsets)
                const unsigned vrow = unsigned(16 * tt + 4 * g) * d + unsigned(min(f, d - 1));
                const uint16_t *vp16 = vu16 + vrow;
                const typename E::T *vp = vu + vrow;
                if constexpr (BFM) {
#pragma unroll
                    for (int pp = 0; pp < 2; ++pp) {
                        u16x2 pr;
                        pr.x = vp16[2 * pp * d];
                        pr.y = vp16[(2 * pp + 1) * d];
                        vh_[u][ct][pp] = __builtin_bit_cast(uint32_t, pr);
                    }
                } else {
#pragma unroll
                    for (int x = 0; x < 4; ++x)
                        vr_[u][ct][x] = E::load(vp, x * d);
                }
            }
        }
    };
    // One pair of key tiles for every landmark tile: ones column, logits,
    // running maxima, G_U^n and T.  The K chunks stay unmasked: their
    // overlapping slots meet zeros in the Qbar slots.
    auto process = [&](int t0, float (&kr_)[2][8], bf8 (&kw_)[2], float (&vr_)[2][NCT][4],
                       uint32_t (&vh_)[2][NCT][2]) {
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                const int f = 16 * ct + c;
                if constexpr (BFM) {
#pragma unroll
                    for (int pp = 0; pp < 2; ++pp)
                        vh_[u][ct][pp] = f < d ? vh_[u][ct][pp]
                                               : (PAD && f == d ? 0x3F803F80u : 0u);
                } else {
#pragma unroll
                    for (int x = 0; x < 4; ++x)
                        vr_[u][ct][x] = f < d ? vr_[u][ct][x] : (PAD && f == d ? 1.f : 0.f);
                }
            }
        const bool second = t0 + 1 < NT;   // uniform
        bf8 vv[NCT];   // bf16 path: V of the pair as the right-hand operand
        if constexpr (BFM) {
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                U16B vb;
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
                    vb.w[jj] = vh_[jj >> 1][ct][jj & 1];
                vv[ct] = __builtin_bit_cast(bf8, vb);
            }
        }
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            // S_U^T tiles: lane (g, c) gets S_U[landmark 16j + c][key 16tt + 4g + i].
            f4 su[2];
            float gmax = -INFINITY;
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                f4 acc = {0.f, 0.f, 0.f, 0.f};
                if constexpr (BFM) {
                    acc = mfma_bf16(kw_[u], qjh[j], acc);
                    acc = mfma_bf16(kw_[u], qjl[j], acc);
                } else {
#pragma unroll
                    for (int x = 0; x < 8; ++x)
                        acc = mfma4(kr_[u][x], qj[j][x], acc);
                }
                su[u] = acc;
                // a repeated last tile (fp32 path, odd tile count) leaves the
                // maximum unchanged, so it needs no exclusion here
                gmax = fmaxf(gmax, fmaxf(fmaxf(acc[0], acc[1]), fmaxf(acc[2], acc[3])));
            }
            const float mnew = fmaxf(mrj[j], max_groups(gmax));
            // Rescale what is accumulated when a maximum grew; the factor is
            // exactly 1 for every landmark whose maximum held, so skipping the
            // step when none grew changes nothing.
            if (__builtin_amdgcn_ballot_w64(mnew != mrj[j]) != 0) {
                const float f = fast_exp2(a.s2 * (mrj[j] - mnew));
                tdj[j] *= f;
                const f4 fr = by_rows(f, vec, g, c);   // factor of landmark 16j + 4g + i
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
                    TJ[j][ct] *= fr;
            }
            mrj[j] = mnew;
            // Landmarks past m get an infinite offset: their terms are exactly 0.
            const float mb = (FULL || 16 * j + c < m) ? a.s2 * mnew : INFINITY;
            if constexpr (BFM) {
                // bf16 product over the 32 keys of the pair, lane group g
                // supplying keys 4g..4g+3 of both tiles (N % 32 == 0 here)
                float gk[8];
#pragma unroll
                for (int h = 0; h < 2; ++h)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        gk[4 * h + i] = fast_exp2(fmaf(a.s2, su[h][i], -mb));
                        if constexpr (!PAD)
                            tdj[j] += gk[4 * h + i];
                    }
                bf8 gh, gl;
                split_bf16(gk, gh, gl);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    TJ[j][ct] = mfma_bf16(gh, vv[ct], TJ[j][ct]);
                    TJ[j][ct] = mfma_bf16(gl, vv[ct], TJ[j][ct]);
                }
            } else {
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    if (u == 1 && !second)
                        break;   // uniform
                    f4 e;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        e[i] = fast_exp2(fmaf(a.s2, su[u][i], -mb));
                        if constexpr (!PAD)
                            tdj[j] += e[i];
                    }
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                        for (int x = 0; x < 4; ++x)
                            TJ[j][ct] = mfma4(e[x], vr_[u][ct][x], TJ[j][ct]);
                }
            }
        }
        if constexpr (KP) {
            // Step 1 for K.  The product K_tile x ksel (tile ct) puts K[token
            // 16tt + 4g + i][feature 16ct + c] in lane (g, c); the tokens 4g..4g+3
            // of a tile are four adjacent columns of one image row, i.e. one
            // patch row.  One tile per row (16 x 16 windows): both tiles of the
            // pair are rows of the same patches, accumulated in one product.
            // Two tiles per row (32 x 32): tile u holds columns 16u.., patches
            // 4u + g.
            constexpr bool one_row_tile = KPL == 1;
            if constexpr (KPL == 1)
                ksel_own = own_selector();
            const f4 z4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ct = 0; ct < 2; ++ct) {
                U16B sw;
#pragma unroll
                for (int pp = 0; pp < 4; ++pp)
                    sw.w[pp] = (g >> 1) == ct ? ksel_own.w[pp] : 0u;
                const bf8 ksel = __builtin_bit_cast(bf8, sw);
                f4 d0 = mfma_bf16(kw_[0], ksel, z4);
                if constexpr (one_row_tile) {
                    d0 = mfma_bf16(kw_[1], ksel, d0);
                } else {
                    const f4 d1 = mfma_bf16(kw_[1], ksel, z4);
                    pk[1][ct] += (d1[0] + d1[1]) + (d1[2] + d1[3]);
                }
                pk[0][ct] += (d0[0] + d0[1]) + (d0[2] + d0[3]);
            }
            const int pair = t0 >> 1;
            if (KPL == 1 || (pair + 1) % ppb == 0) {   // uniform: the band is complete
                const int band = KPL == 1 ? pair : pair / ppb;
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    if (u == 1 && one_row_tile)
                        break;   // compile-time
                    const int lk = band * a.gc + 4 * u + g;
#pragma unroll
                    for (int ct = 0; ct < 2; ++ct) {
                        if (16 * ct + c < D)
                            kbar[lk * kTS + 16 * ct + c] = pk[u][ct] * a.inv_patch;
                        pk[u][ct] = 0.f;
                    }
                }
            }
        }
    };
    // Unrolled by two with two buffers (no loaded row is copied) where the
    // registers allow it; bf16 with three or four landmark tiles copies the
    // prefetched pair instead.
    load_pair(t_begin, kr, kw, vr, vh);
    if constexpr (!(BFM && MT >= 3)) {
        for (int t0 = t_begin; t0 < t_end; t0 += 2 * t_stride) {
            load_pair(t0 + t_stride, krn, kwn, vrn, vhn);
            process(t0, kr, kw, vr, vh);
            if (t0 + t_stride >= t_end)
                break;   // uniform
            load_pair(t0 + 2 * t_stride, kr, kw, vr, vh);
            process(t0 + t_stride, krn, kwn, vrn, vhn);
        }
    } else {
        for (int t0 = t_begin; t0 < t_end; t0 += t_stride) {
            load_pair(t0 + t_stride, krn, kwn, vrn, vhn);
            process(t0, kr, kw, vr, vh);
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                kw[u] = kwn[u];
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                    for (int x = 0; x < 2; ++x)
                        vh[u][ct][x] = vhn[u][ct][x];
            }
        }
    }
    // This wave's record: T rows of every landmark, T_D and the maxima.  An
    // idle wave (fewer key pairs than waves) leaves -inf maxima, which the
    // merge weighs by exp2(-inf) = 0.
    {
        float *rw = lds + L::recs + lt * L::rec_len;
#pragma unroll
        for (int j = 0; j < MT; ++j) {
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    rw[(16 * j + 4 * g + i) * kRecP + 16 * ct + c] = TJ[j][ct][i];
            const float td = PAD ? 0.f : sum_groups(tdj[j]);
            if (g == 0) {
                rw[LD + 16 * j + c] = td;
                rw[LM + 16 * j + c] = mrj[j];
            }
        }
    }
    __syncthreads();
    // Merge for this wave's landmark tile lt: m_U = the largest of the
    // waves' maxima; T and T_D = sum over waves of exp(s (max_w - m_U)) x
    // the wave's sums.
    f4 T[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
    float tden = 0.f, mrun = -INFINITY;
    f4 mrows = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};   // m_U of landmarks 16lt+4g+i
    {
        const float *rb = lds + L::recs;
#pragma unroll
        for (int w = 0; w < MT; ++w) {
            const float *rw = rb + w * L::rec_len;
            mrun = fmaxf(mrun, rw[LM + l]);
            const f4 mw = *reinterpret_cast<const f4 *>(rw + LM + 16 * lt + 4 * g);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                mrows[i] = fmaxf(mrows[i], mw[i]);
        }
#pragma unroll
        for (int w = 0; w < MT; ++w) {
            const float *rw = rb + w * L::rec_len;
            const float fl = fast_exp2(a.s2 * (rw[LM + l] - mrun));   // 0 for an idle wave
            tden = fmaf(fl, PAD ? rw[(16 * lt + c) * kRecP + D] : rw[LD + l], tden);
            const f4 mw = *reinterpret_cast<const f4 *>(rw + LM + 16 * lt + 4 * g);
            f4 fr;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                fr[i] = fast_exp2(a.s2 * (mw[i] - mrows[i]));
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                f4 x;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    x[i] = rw[(16 * lt + 4 * g + i) * kRecP + 16 * ct + c];
                T[ct] += fr * x;
            }
        }
    }
    const float mu = a.s2 * mrun;   // m_U of landmark l (base-2 units)

    // This lane's Qbar row, read back from its table (intact until the core
    // overwrites the region, after its first barrier) rather than held in
    // registers through the key pass: fewer registers for the fp32 and KP
    // kernels (c4 fp32 -0.8%); the bf16 kernel without KP keeps its registers
    // (+0.4% with the reload).
    float qbl[8];
#pragma unroll
    for (int s = 0; s < 8; ++s) {
        if constexpr (KP || !BFM)
            qbl[s] = slot_valid<D>(g, s) ? qtab[l * kTS + chunk_start<D>(g) + s] : 0.f;
        else
            qbl[s] = qb[s];
    }
    landmark_core<MT, D, BFM, FULL>(lds, qbl, mu, T, tden, m, a.iters, a.s2, lt, lane);
    constexpr int TDo = table_den<MT>();
    float *Wb = lds + L::wb;

    // ---- Steps 3 (G_L side), 6 and 7 over this wave's token tiles.
    constexpr int MP = (MT + 1) / 2;   // landmark tile pairs (bf16 path)
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
    // bf16 path: Kbar rows and W as hi + lo terms.  W pairs landmark tiles
    // (2kp, 2kp+1): lane group g supplies landmarks 4g..4g+3 of both.
    bf8 kbh[MT], kbl[MT], wh[MP][2], wl[MP][2];
    if constexpr (BFM) {
#pragma unroll
        for (int kk = 0; kk < MT; ++kk)
            split_bf16(kb[kk], kbh[kk], kbl[kk]);
#pragma unroll
        for (int kp = 0; kp < MP; ++kp)
#pragma unroll
            for (int ct = 0; ct < 2; ++ct) {
                float w8[8];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    w8[i] = WR[2 * kp][ct][i];
                    w8[4 + i] = (2 * kp + 1 < MT) ? WR[(2 * kp + 1) % MT][ct][i] : 0.f;
                }
                split_bf16(w8, wh[kp][ct], wl[kp][ct]);
            }
    }
    const uint16_t *qu16 = reinterpret_cast<const uint16_t *>(qu);
    // Token tiles of this wave: lt, lt + MT, ...; the Q rows of kQGroup tiles
    // loaded together; the next group's rows are requested before this group
    // is computed (as in the key pass).  The chunks stay unmasked: the
    // overlapping slots meet zeros on the Kbar side.
    constexpr int kQGroup = 2;
    float qg[kQGroup][8], qgn[kQGroup][8];
    bf8 qw[kQGroup], qwn[kQGroup];
    auto load_q = [&](int t0, float (&qg_)[kQGroup][8], bf8 (&qw_)[kQGroup]) {
#pragma unroll
        for (int u = 0; u < kQGroup; ++u) {
            const int64_t row = int64_t(16 * min(t0 + u * MT, NT - 1) + c) * d;
            if constexpr (BFM)
                qw_[u] = load_row8_bf16(qu16 + row + chunk_start<D>(g));
            else if constexpr (E::bytes == 4)
                load_row8<D>(qu + row + chunk_start<D>(g), qg_[u]);
            else
                load_chunk8<E, D>(qu + row, g, qg_[u]);
        }
    };
    load_q(lt, qg, qw);
    for (int t0 = lt; t0 < NT; t0 += kQGroup * MT) {
        load_q(t0 + kQGroup * MT, qgn, qwn);
#pragma unroll
        for (int u = 0; u < kQGroup; ++u) {
            const int tt = t0 + u * MT;
            if (tt >= NT)
                break;   // uniform
            f4 glT[MT];   // lane (g,c): G_L^n[token 16tt+c][landmark 16kk+4g+i]
            float ml = -INFINITY;
#pragma unroll
            for (int kk = 0; kk < MT; ++kk) {
                f4 acc = {0.f, 0.f, 0.f, 0.f};
                if constexpr (BFM) {
                    acc = mfma_bf16(kbh[kk], qw[u], acc);
                    acc = mfma_bf16(kbl[kk], qw[u], acc);
                } else {
#pragma unroll
                    for (int s = 0; s < 8; ++s)
                        acc = mfma4(kb[kk][s], qg[u][s], acc);
                }
                glT[kk] = acc;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (FULL || 16 * kk + 4 * g + i < m)
                        ml = fmaxf(ml, acc[i]);
            }
            ml = a.s2 * max_groups(ml);
            float od = 0.f;
#pragma unroll
            for (int kk = 0; kk < MT; ++kk)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float e = (FULL || 16 * kk + 4 * g + i < m)
                                        ? fast_exp2(fmaf(a.s2, glT[kk][i], -ml)) : 0.f;
                    glT[kk][i] = e;
                    if constexpr (!PAD)
                        od = fmaf(e, wdv[kk][i], od);
                }
            f4 rcp;   // 1 / O_D[16tt + 4g + i]
            if constexpr (!PAD) {
                od = sum_groups(od);
                const f4 odr = by_rows(od, vec, g, c);
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    rcp[i] = __builtin_amdgcn_rcpf(odr[i]);
            }
            bf8 gh[MP], gl[MP];
            if constexpr (BFM) {
#pragma unroll
                for (int kp = 0; kp < MP; ++kp) {
                    float g8[8];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        g8[i] = glT[2 * kp][i];
                        g8[4 + i] = (2 * kp + 1 < MT) ? glT[(2 * kp + 1) % MT][i] : 0.f;
                    }
                    split_bf16(g8, gh[kp], gl[kp]);
                }
            }
            f4 ont[2];
#pragma unroll
            for (int ct = 0; ct < 2; ++ct) {
                f4 on = {0.f, 0.f, 0.f, 0.f};
                if constexpr (BFM) {
#pragma unroll
                    for (int kp = 0; kp < MP; ++kp) {
                        on = mfma_bf16(gh[kp], wh[kp][ct], on);
                        on = mfma_bf16(gh[kp], wl[kp][ct], on);
                        on = mfma_bf16(gl[kp], wh[kp][ct], on);
                    }
                } else {
#pragma unroll
                    for (int kk = 0; kk < MT; ++kk)
                        on = mm16_acc(glT[kk], WR[kk][ct], on);
                }
                ont[ct] = on;
            }
            if constexpr (PAD) {
                // O_D is column D: lane D % 16 of each row of feature tile D / 16
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    rcp[i] = __builtin_amdgcn_rcpf(row_bcast<D % 16>(ont[D / 16][i]));
            }
#pragma unroll
            for (int ct = 0; ct < 2; ++ct) {
                const f4 on = ont[ct];
                const int f = 16 * ct + c;
                if (f < d) {
                    const int64_t orow = int64_t(16 * tt + 4 * g) * d + f;
                    if constexpr (E::bytes == 2) {
                        // rows (0, 1) and (2, 3) converted in pairs (round to
                        // nearest even), stored as 16-bit values
                        uint16_t *o16 = reinterpret_cast<uint16_t *>(ou) + orow;
                        const uint32_t p01 = cvt_bf16x2(on[0] * rcp[0], on[1] * rcp[1]);
                        const uint32_t p23 = cvt_bf16x2(on[2] * rcp[2], on[3] * rcp[3]);
                        o16[0] = uint16_t(p01);
                        o16[d] = uint16_t(p01 >> 16);
                        o16[2 * d] = uint16_t(p23);
                        o16[3 * d] = uint16_t(p23 >> 16);
                    } else {
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            E::store(ou, orow + i * d, on[i] * rcp[i]);
                    }
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kQGroup; ++u) {
            qw[u] = qwn[u];
#pragma unroll
            for (int x = 0; x < 8; ++x)
                qg[u][x] = qgn[u][x];
        }
    }
}

// bf16 inputs with N % 32 == 0 take the bf16 matrix-core path.
// K pooled in the key pass: square windows one or two 16-token tiles wide,
// patches four tokens wide (a patch row is one lane group's four tokens of a
// tile), whole bands of patches per wave.
bool kpool_ok(const Problem &p, int MT)
{
    const Geometry &g = p.geo;
    if (g.rows != g.cols || g.rows * g.cols != p.N || g.pc != 4 || (g.cols != 16 && g.cols != 32))
        return false;
    const int tpr = g.cols / 16, pairs = p.N / 32;
    if ((g.pr * tpr) % 2 != 0 || pairs % MT != 0)
        return false;
    return (pairs / MT) % (g.pr * tpr / 2) == 0;
}

template <class E, int MT, int D, bool FULL>
void launch_large_f(const Problem &p, const LargeArgs &a, hipStream_t stream)
{
    const size_t lds = size_t(LargeLds<MT>::total) * sizeof(float);
    const auto *q = static_cast<const typename E::T *>(p.q);
    const auto *k = static_cast<const typename E::T *>(p.k);
    const auto *v = static_cast<const typename E::T *>(p.v);
    auto *o = static_cast<typename E::T *>(p.o);
    const dim3 grid(unsigned(p.units)), block(64 * MT);
    if (E::bytes == 2 && p.N % 32 == 0) {
        // KP for two landmark tiles (16 x 16 windows, m = 32, 2 x 4 patches) and
        // four (32 x 32, m = 64, 4 x 4 patches); other shapes keep the pooling
        // loop.
        if constexpr (E::bytes == 2 && FULL && MT == 2) {
            if (kpool_ok(p, MT) && p.geo.cols == 16 && p.geo.pr == 2) {
                hipLaunchKernelGGL((tiled_large_kernel<E, MT, D, true, true, 1>), grid, block,
                                   lds, stream, q, k, v, o, a);
                return;
            }
        }
        if constexpr (E::bytes == 2 && FULL && MT == 4) {
            if (kpool_ok(p, MT) && p.geo.cols == 32) {
                hipLaunchKernelGGL((tiled_large_kernel<E, MT, D, true, true, 2>), grid, block,
                                   lds, stream, q, k, v, o, a);
                return;
            }
        }
        hipLaunchKernelGGL((tiled_large_kernel<E, MT, D, E::bytes == 2, FULL, 0>), grid,
                           block, lds, stream, q, k, v, o, a);
    } else {
        hipLaunchKernelGGL((tiled_large_kernel<E, MT, D, false, FULL, 0>), grid, block, lds,
                           stream, q, k, v, o, a);
    }
}

template <class E, int MT, int D>
void launch_large(const Problem &p, const LargeArgs &a, hipStream_t stream)
{
    if (p.m == 16 * MT)
        launch_large_f<E, MT, D, true>(p, a, stream);
    else
        launch_large_f<E, MT, D, false>(p, a, stream);
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
    case 12: launch_large_m<E, 12>(p, a, stream); break;
    case 16: launch_large_m<E, 16>(p, a, stream); break;
    case 20: launch_large_m<E, 20>(p, a, stream); break;
    case 24: launch_large_m<E, 24>(p, a, stream); break;
    case 28: launch_large_m<E, 28>(p, a, stream); break;
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
