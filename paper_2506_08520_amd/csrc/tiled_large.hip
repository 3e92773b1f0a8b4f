// MFMA-tiled PnP-Nystra kernel for large windows (N a multiple of 16, e.g.
// 16x16 and 32x32 windows; m <= 64 landmarks; d_h in {8, 12, ..., 28, 30, 32}).
//
// One workgroup computes one (window, head) unit with MT = ceil(m / 16)
// wavefronts; wave w owns landmark tile w (landmarks 16w .. 16w+15):
//   1. Step 1: each lane averages the patch of its own landmark straight from
//      global memory (any pooling grid), producing Qbar rows in registers and
//      Kbar rows in LDS.
//   2. Step 3, G_U side: the wave streams all N keys once, keeping the row
//      maxima m_U of its landmarks as running maxima and accumulating
//      G_U^n and T = G_U^n [V | 1], rescaled whenever a maximum grows.
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
template <class E, int MT, int D, bool BFM, bool FULL>
__global__ void __launch_bounds__(64 * MT)
tiled_large_kernel(const typename E::T *__restrict__ q, const typename E::T *__restrict__ k,
                   const typename E::T *__restrict__ v, typename E::T *__restrict__ o,
                   LargeArgs a)
{
    using L = LargeLds<MT>;
    constexpr int d = D;
    // With a spare column (D % 16 != 0), column D of V is replaced by ones, so
    // that column D of T, W and O carries T_D, W_D and O_D (no separate sums).
    constexpr bool PAD = D % 16 != 0;
    extern __shared__ float lds[];
    float *kbar = lds + L::kbar;

    const int lt = threadIdx.x >> 6, lane = threadIdx.x & 63;
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
        const int le = lval ? l : m - 1;   // padding lanes read a valid patch, then drop it
        const int r0 = (le / a.gc) * a.pr, c0 = (le % a.gc) * a.pc;
        const int npatch = a.pr * a.pc;
        // Rows arrive raw; the slots a lower lane group carries are zeroed
        // once, in the sums (the same values as zeroing every row).
        constexpr int kP = 8;
        for (int j0 = 0; j0 < npatch; j0 += kP) {
            float x[kP][8], y[kP][8];   // fp32 rows
            U16B xb[kP], yb[kP];        // bf16 rows (raw pairs)
#pragma unroll
            for (int u = 0; u < kP; ++u) {
                const int j = min(j0 + u, npatch - 1);
                const int64_t t = (int64_t(r0 + j / a.pc) * a.cols + c0 + j % a.pc) * d +
                                  chunk_start<D>(g);
                if constexpr (E::bytes == 4) {
                    load_row8<D>(qu + t, x[u]);
                    load_row8<D>(ku + t, y[u]);
                } else {
                    xb[u] = *reinterpret_cast<const U16B *>(qu + t);
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
                            kbv[2 * w] += __uint_as_float(yb[u].w[w] << 16);
                            kbv[2 * w + 1] += __uint_as_float(yb[u].w[w] & 0xffff0000u);
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
#pragma unroll
    for (int s = 0; s < 8; ++s)
        if (slot_valid<D>(g, s))
            kbar[l * kTS + chunk_start<D>(g) + s] = kbv[s];

    // ---- Step 3, G_U side, one pass over the N keys, kGroup key tiles per
    // step: m_U of this landmark as a running maximum, and G_U^n and
    // T = G_U^n [V | 1] accumulated against it; when the maximum grows, the
    // partial T and T_D are rescaled by exp(old - new), so that at the end they
    // hold exactly the sums against the final m_U.
    constexpr int kGroup = 4;
    const uint16_t *ku16 = reinterpret_cast<const uint16_t *>(ku);
    bf8 qbh, qbl;   // bf16 path: Qbar row as hi + lo terms
    if constexpr (BFM)
        split_bf16(qb, qbh, qbl);
    // S_U^T tile for key tile tt: lane (g,c) gets S_U[landmark l][key 16tt + 4g + i].
    auto su_tile = [&](int tt, const float *kr, const bf8 &kraw) {
        f4 acc = {0.f, 0.f, 0.f, 0.f};
        if constexpr (BFM) {
            acc = mfma_bf16(kraw, qbh, acc);
            acc = mfma_bf16(kraw, qbl, acc);
        } else {
#pragma unroll
            for (int s = 0; s < 8; ++s)
                acc = mfma4(kr[s], qb[s], acc);
        }
        return acc;
    };
    // T[ct] lane (g,c): T[landmark 16lt+4g+i][feature 16ct+c].
    f4 T[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
    float tden = 0.f;    // this lane's share of T_D of landmark l
    float mrun = -INFINITY;   // running max of S_U[l][.] (unscaled logits)
    const uint16_t *vu16 = reinterpret_cast<const uint16_t *>(vu);
    // Key groups are software-pipelined: the loads of group t0 + kGroup are
    // issued before group t0 is computed (past the end they repeat the last
    // tile and go unused).  Chunks are loaded raw, so no instruction waits on
    // a load at its issue.
    // bf16 V is held as pairs of rows (4g, 4g+1) and (4g+2, 4g+3) of one
    // column, the two 16-bit loads landing in the halves of one register.
    typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
    float kr[kGroup][8], vr[kGroup][2][4], krn[kGroup][8], vrn[kGroup][2][4];
    bf8 kw[kGroup], kwn[kGroup];
    uint32_t vh[kGroup][2][2], vhn[kGroup][2][2];
    auto load_group = [&](int t0, float (&kr_)[kGroup][8], bf8 (&kw_)[kGroup],
                          float (&vr_)[kGroup][2][4], uint32_t (&vh_)[kGroup][2][2]) {
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
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
            for (int ct = 0; ct < 2; ++ct) {
                const int f = 16 * ct + c;
                // Columns past d repeat column d - 1: they reach only columns
                // of T, W and O that are never stored (T_D is summed apart).
                // one address per row group; the four rows are immediate offsets
                const unsigned vrow = unsigned(16 * tt + 4 * g) * d + unsigned(min(f, d - 1));
                const uint16_t *vp16 = vu16 + vrow;
                const typename E::T *vp = vu + vrow;
                if constexpr (BFM) {
#pragma unroll
                    for (int p = 0; p < 2; ++p) {
                        u16x2 pr;
                        pr.x = vp16[2 * p * d];
                        pr.y = vp16[(2 * p + 1) * d];
                        vh_[u][ct][p] = __builtin_bit_cast(uint32_t, pr);
                    }
                } else {
#pragma unroll
                    for (int s = 0; s < 4; ++s)
                        vr_[u][ct][s] = E::load(vp, s * d);
                }
            }
        }
    };
    // One group of key tiles: masks, logits, running maxima, G_U^n and T.
    // The K chunks stay unmasked: their overlapping slots meet zeros in the
    // Qbar slots (Step 1 zeroes them).
    auto process = [&](int t0, float (&kr)[kGroup][8], bf8 (&kw)[kGroup],
                       float (&vr)[kGroup][2][4], uint32_t (&vh)[kGroup][2][2]) {
        if constexpr (PAD) {
            const bool ones = c == D % 16;   // column D, in feature tile D / 16
#pragma unroll
            for (int u = 0; u < kGroup; ++u) {
                if constexpr (BFM) {
#pragma unroll
                    for (int p = 0; p < 2; ++p)
                        vh[u][D / 16][p] = ones ? 0x3F803F80u : vh[u][D / 16][p];   // bf16 1.0, twice
                } else {
#pragma unroll
                    for (int x = 0; x < 4; ++x)
                        vr[u][D / 16][x] = ones ? 1.f : vr[u][D / 16][x];
                }
            }
        }
        // Logits of the group (a repeated last tile leaves the maximum unchanged
        // and is not accumulated).
        f4 su[kGroup];
        float gmax = -INFINITY;
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
            su[u] = su_tile(min(t0 + u, NT - 1), kr[u], kw[u]);
            gmax = fmaxf(gmax, fmaxf(fmaxf(su[u][0], su[u][1]), fmaxf(su[u][2], su[u][3])));
        }
        const float mnew = fmaxf(mrun, max_groups(gmax));
        {   // rescale what is accumulated: factor 1 exactly when the maximum
            // holds, 0 on the first group (all lanes take part in the exchange)
            const float f = fast_exp2(a.s2 * (mrun - mnew));
            tden *= f;
            const f4 fr = by_rows(f, vec, g, c);   // factor of landmark 16lt+4g+i
            T[0] *= fr;
            T[1] *= fr;
        }
        mrun = mnew;
        const float mb = a.s2 * mnew;
        if constexpr (BFM) {
            // Key tiles in pairs: the bf16 product contracts 32 keys, lane group g
            // supplying keys 4g..4g+3 of both tiles.  N % 32 == 0 on this path.
#pragma unroll
            for (int u = 0; u < kGroup; u += 2) {
                if (t0 + u >= NT)
                    break;   // uniform
                float gk[8];
#pragma unroll
                for (int h = 0; h < 2; ++h)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        gk[4 * h + i] = lval ? fast_exp2(fmaf(a.s2, su[u + h][i], -mb)) : 0.f;
                        if constexpr (!PAD)
                            tden += gk[4 * h + i];
                    }
                bf8 gh, gl;
                split_bf16(gk, gh, gl);
#pragma unroll
                for (int ct = 0; ct < 2; ++ct) {
                    U16B vb;
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        vb.w[j] = vh[u + (j >> 1)][ct][j & 1];
                    const bf8 vv = __builtin_bit_cast(bf8, vb);
                    T[ct] = mfma_bf16(gh, vv, T[ct]);
                    T[ct] = mfma_bf16(gl, vv, T[ct]);
                }
            }
        } else {
#pragma unroll
            for (int u = 0; u < kGroup; ++u) {
                if (t0 + u >= NT)
                    break;   // uniform
                f4 e;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    e[i] = lval ? fast_exp2(fmaf(a.s2, su[u][i], -mb)) : 0.f;
                    if constexpr (!PAD)
                        tden += e[i];
                }
#pragma unroll
                for (int ct = 0; ct < 2; ++ct)
#pragma unroll
                    for (int s = 0; s < 4; ++s)
                        T[ct] = mfma4(e[s], vr[u][ct][s], T[ct]);
            }
        }
    };
    // Unrolled by two with two buffers, so that no loaded row is copied.
    load_group(0, kr, kw, vr, vh);
    for (int t0 = 0; t0 < NT; t0 += 2 * kGroup) {
        load_group(t0 + kGroup, krn, kwn, vrn, vhn);
        process(t0, kr, kw, vr, vh);
        if (t0 + kGroup >= NT)
            break;   // uniform
        load_group(t0 + 2 * kGroup, kr, kw, vr, vh);
        process(t0 + kGroup, krn, kwn, vrn, vhn);
    }
    const float mu = a.s2 * mrun;   // m_U of landmark l (base-2 units)
    // T_D of landmark l (with the ones column it is column D of T, and the
    // core's separate W_D goes unused)
    if constexpr (!PAD)
        tden = sum_groups(tden);
    __syncthreads();           // Kbar complete

    landmark_core<MT, D, BFM, FULL>(lds, qb, mu, T, tden, m, a.iters, a.s2, lt, lane);
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
template <class E, int MT, int D, bool FULL>
void launch_large_f(const Problem &p, const LargeArgs &a, hipStream_t stream)
{
    const size_t lds = size_t(LargeLds<MT>::total) * sizeof(float);
    const auto *q = static_cast<const typename E::T *>(p.q);
    const auto *k = static_cast<const typename E::T *>(p.k);
    const auto *v = static_cast<const typename E::T *>(p.v);
    auto *o = static_cast<typename E::T *>(p.o);
    const dim3 grid(unsigned(p.units)), block(64 * MT);
    if (E::bytes == 2 && p.N % 32 == 0)
        hipLaunchKernelGGL((tiled_large_kernel<E, MT, D, E::bytes == 2, FULL>), grid, block,
                           lds, stream, q, k, v, o, a);
    else
        hipLaunchKernelGGL((tiled_large_kernel<E, MT, D, false, FULL>), grid, block, lds,
                           stream, q, k, v, o, a);
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
