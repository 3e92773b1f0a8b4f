// Token-split PnP-Nystra: Algorithm 1 as six launches over a caller-provided
// workspace, for windows so large, or (window, head) units so few, that one
// workgroup per unit leaves most of the 256 compute units idle -- global
// attention, where one window is the whole feature map, is the extreme case.
//
//   A   pool     grid units x m x pieces: sums of Q and K over one piece of
//                one landmark's pooling patch (Step 1).
//   A2  bar      grid units: Qbar, Kbar = piece sums / patch size.
//   B   keys     grid units x key chunks: per chunk and landmark, the maximum
//                of S_U over the chunk's keys and T = G_U [V | 1] against it
//                (Step 3, G_U side), the four waves merged in LDS.
//   C   merge    grid units x landmark tiles x 9 column groups: the chunk
//                records merged to m_U = max over chunks and
//                T = sum_c exp(s (max_c - m_U)) T_c (same for T_D), the sums
//                of Step 3 against the global row maximum.
//   P   core     grid units: Steps 2, 4 and 5-6 (landmark_core).
//   D   queries  grid units x query chunks: Steps 3 (G_L side), 6 and 7.
//
// Only the order of the additions differs from the one-pass kernels.  Q is
// read twice (A, D), K twice (A, B), V once; O is written once.  Every
// contraction of B and D runs on the matrix cores exactly as in the one-pass
// large kernel (fp32, or bf16 with hi + lo terms for bf16 inputs).
#include "internal.hpp"
#include "core_tiles.hpp"

namespace nystra {
namespace {

using namespace tile;
using namespace core;

constexpr int kWP = 32;                    // pitch (floats) of feature rows in the workspace
constexpr int kLm = 64;                    // landmark rows reserved per unit
// Chunk record of pass B: T by column groups of four ([kWP / 4][kLm][4], so a
// merge block reads one contiguous piece per chunk), then T_D, then the row
// maxima.  The merged record of pass C has T row-major ([kLm][kWP]) instead.
constexpr int kRecT = kLm * kWP;
constexpr int kRecD = kRecT;
constexpr int kRecM = kRecT + kLm;
constexpr int kRec = kRecT + 2 * kLm;
constexpr int kWout = kLm * kTS + kLm;     // W table (pitch kTS) and W_D
constexpr int kWaves = 4;                  // waves per workgroup of passes A, B, D
constexpr int kMergeGroups = kWP / 4 + 1;  // column groups of pass C (8 x 4 features, T_D)

struct SplitArgs {
    int64_t units;
    int N, d, m, iters;
    float s2;          // logit scale in base-2 units (scale * log2 e)
    float inv_patch;   // 1 / tokens per pooling patch
    int cols, pr, pc, gc;
    int P;             // tokens per patch
    int pieces, piece_len;     // pass A: pieces per patch, tokens per piece
    int nchunk, chunk_len;     // pass B: key chunks per unit, keys per chunk
    int nqchunk, qchunk_len;   // pass D: query chunks per unit, queries per chunk
    float *part;   // [units][2][m * pieces][kWP]  piece sums of Q, then K
    float *bar;    // [units][2][kLm][kWP]         Qbar, then Kbar (zero past m, d)
    float *rec;    // [units][nchunk][kRec]        chunk records of pass B (T by column groups)
    float *comb;   // [units][kRec]                merged T, T_D and s2 * m_U
    float *wout;   // [units][kWout]               W and W_D
};

__device__ inline int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// ---- A: piece sums of Q and K ------------------------------------------------
template <class E, int D>
__global__ void __launch_bounds__(64 * kWaves)
split_pool_kernel(const typename E::T *__restrict__ q, const typename E::T *__restrict__ k,
                  SplitArgs a)
{
    __shared__ float red[kWaves][2][4][8];
    const int per_unit = a.m * a.pieces;
    const int64_t unit = blockIdx.x / per_unit;
    const int rem = int(blockIdx.x - unit * per_unit);
    const int l = rem / a.pieces, r = rem - l * a.pieces;
    const int i0 = r * a.piece_len, i1 = min(a.P, i0 + a.piece_len);
    const int w = wave_id(), lane = threadIdx.x & 63, g = lane >> 4, c = lane & 15;
    const int r0 = (l / a.gc) * a.pr, c0 = (l % a.gc) * a.pc;
    const int64_t base = unit * int64_t(a.N) * D;
    const typename E::T *qu = q + base, *ku = k + base;

    float qs[8], ks[8];
#pragma unroll
    for (int s = 0; s < 8; ++s)
        qs[s] = ks[s] = 0.f;
    // Wave w takes 16-token tiles w, w + 4, ... of the piece; four tiles per
    // step so that their loads are in flight together.  When patch rows and
    // pieces are whole tiles (pc and the piece length multiples of 16), a
    // tile is 16 consecutive tokens of one patch row: its position is
    // computed once per tile (uniform, scalar) instead of per lane.
    const bool whole_tiles = a.pc % 16 == 0 && a.piece_len % 16 == 0;   // uniform
    for (int b = i0 + 16 * w; b < i1; b += 4 * 16 * kWaves) {
        float x[4][8], y[4][8];
        bool ok[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            int64_t t;
            if (whole_tiles) {
                const int ib = b + 16 * kWaves * u;   // tile start, uniform
                ok[u] = ib < i1;
                const int ii = ok[u] ? ib : i0;
                t = int64_t(r0 + ii / a.pc) * a.cols + c0 + ii % a.pc + c;
            } else {
                const int i = b + 16 * kWaves * u + c;
                ok[u] = i < i1;
                const int ii = ok[u] ? i : i0;
                t = int64_t(r0 + ii / a.pc) * a.cols + c0 + ii % a.pc;
            }
            load_chunk8<E, D>(qu + t * D, g, x[u]);
            load_chunk8<E, D>(ku + t * D, g, y[u]);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (ok[u]) {
#pragma unroll
                for (int s = 0; s < 8; ++s) {
                    qs[s] += x[u][s];
                    ks[s] += y[u][s];
                }
            }
    }
#pragma unroll
    for (int s = 0; s < 8; ++s) {
        qs[s] = sum_row(qs[s]);   // every lane of the row holds the sum
        ks[s] = sum_row(ks[s]);
    }
    if (c == 0) {
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            red[w][0][g][s] = qs[s];
            red[w][1][g][s] = ks[s];
        }
    }
    __syncthreads();
    if (w == 0) {
        // lane (g, c): tensor c >> 3, slot c & 7 of feature group g
        const int which = c >> 3, s = c & 7;
        float acc = 0.f;
#pragma unroll
        for (int v = 0; v < kWaves; ++v)
            acc += red[v][which][g][s];
        if (slot_valid<D>(g, s)) {
            float *row = a.part + ((unit * 2 + which) * per_unit + rem) * kWP;
            row[chunk_start<D>(g) + s] = acc;
        }
    }
}

// ---- A2: Qbar and Kbar -----------------------------------------------------
// One wave per row (unit, tensor, landmark < kLm): the two halves of the wave
// add alternate pieces, then each other's sums.  Rows past m are zero.
__global__ void __launch_bounds__(64) split_bar_kernel(SplitArgs a)
{
    const int64_t row = blockIdx.x;   // (unit * 2 + which) * kLm + l
    const int l = int(row % kLm);
    const int64_t uw = row / kLm;     // unit * 2 + which
    const int half = threadIdx.x >> 5, f = threadIdx.x & 31;
    float acc = 0.f;
    if (l < a.m && f < a.d) {
        // eight pieces per step, their loads in flight together (the last
        // step's missing pieces read piece `half` and add zero)
        const float *p = a.part + (uw * a.m + l) * int64_t(a.pieces) * kWP + f;
        for (int r0 = half; r0 < a.pieces; r0 += 16) {
            float x[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int r = r0 + 2 * u;
                const float y = p[int64_t(r < a.pieces ? r : half) * kWP];
                x[u] = r < a.pieces ? y : 0.f;
            }
#pragma unroll
            for (int u = 0; u < 8; ++u)
                acc += x[u];
        }
    }
    acc += __shfl_xor(acc, 32, 64);
    if (half == 0)
        a.bar[row * kWP + f] = (l < a.m && f < a.d) ? acc * a.inv_patch : 0.f;
}

// ---- B: chunk records of the G_U side ----------------------------------------
// With d_h % 16 != 0 the first padding column of V is set to 1, so T_D
// accumulates on the matrix cores as column d_h of T; NCT feature tiles of
// 16 columns cover the features (and that column).
template <class E, int MT, int D, bool BFM>
__global__ void __launch_bounds__(64 * kWaves)
split_keys_kernel(const typename E::T *__restrict__ k, const typename E::T *__restrict__ v,
                  SplitArgs a)
{
    constexpr int d = D;
    constexpr bool kOnes = D % 16 != 0;
    constexpr int NCT = (D + 15) / 16;
    // per-wave records in LDS: T rows of the MT tiles, then T_D, then maxima
    constexpr int RR = 16 * MT, LD = RR * kWP, LM = LD + RR, LREC = LD + 2 * RR;
    __shared__ __align__(16) float recs[kWaves][LREC];
    __shared__ float vecs[kWaves][64];
    const int64_t unit = blockIdx.x / a.nchunk;
    const int chunk = int(blockIdx.x - unit * a.nchunk);
    const int w = wave_id(), lane = threadIdx.x & 63, g = lane >> 4, c = lane & 15;
    float *vec = vecs[w];
    const int m = a.m;
    const int64_t base = unit * int64_t(a.N) * d;
    const typename E::T *ku = k + base, *vu = v + base;
    const uint16_t *ku16 = reinterpret_cast<const uint16_t *>(ku);
    const uint16_t *vu16 = reinterpret_cast<const uint16_t *>(vu);
    const float *qbar = a.bar + unit * 2 * kLm * kWP;

    // Qbar rows: lane (g, c) holds landmark 16j + c, the slots of group g.
    float qb[MT][8];
    bf8 qbh[MT], qbl[MT];
#pragma unroll
    for (int j = 0; j < MT; ++j) {
#pragma unroll
        for (int s = 0; s < 8; ++s)
            qb[j][s] = slot_valid<D>(g, s) ? qbar[(16 * j + c) * kWP + chunk_start<D>(g) + s]
                                           : 0.f;
        if constexpr (BFM)
            split_bf16(qb[j], qbh[j], qbl[j]);
    }

    f4 T[MT][NCT];
    float tden[MT], mrun[MT];
#pragma unroll
    for (int j = 0; j < MT; ++j) {
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
            T[j][ct] = f4{0.f, 0.f, 0.f, 0.f};
        tden[j] = 0.f;
        mrun[j] = -INFINITY;
    }
    const int k0 = chunk * a.chunk_len, k1 = min(a.N, k0 + a.chunk_len);
    const int NT = (k1 - k0) >> 4;   // key tiles of the chunk
    // Wave w takes the tile pairs w, w + 4, ...; the second tile of a pair past
    // the chunk's end (fp32 path with an odd tile count) repeats the first and
    // is not accumulated.
    // The pairs are software-pipelined: the next pair's K and V rows are
    // requested before this pair is computed (past the end they repeat the
    // last tile, unused).  Rows arrive raw and the ones column is applied
    // when the pair is consumed, so no instruction waits on a load at its
    // issue.
    // bf16 V is held as pairs of rows (4g, 4g+1) and (4g+2, 4g+3) of one
    // column, the two 16-bit loads landing in the halves of one register.
    typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
    float kr[2][8], vr[2][NCT][4], krn[2][8], vrn[2][NCT][4];
    bf8 kw[2], kwn[2];
    uint32_t vh[2][NCT][2], vhn[2][NCT][2];
    auto load_pair = [&](int t0, float (&kr_)[2][8], bf8 (&kw_)[2], float (&vr_)[2][NCT][4],
                         uint32_t (&vh_)[2][NCT][2]) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int tt = min(t0 + u, NT - 1);
            const int64_t row = int64_t(k0 + 16 * tt + c) * d;
            if constexpr (BFM)
                kw_[u] = load_row8_bf16(ku16 + row + chunk_start<D>(g));
            else if constexpr (E::bytes == 4)
                load_row8<D>(ku + row + chunk_start<D>(g), kr_[u]);
            else   // bf16 values through the fp32 path: unpacked (and masked) here
                load_chunk8<E, D>(ku + row, g, kr_[u]);
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                const int f = 16 * ct + c;
                const int64_t vrow = int64_t(k0 + 16 * tt + 4 * g) * d + min(f, d - 1);
                const uint16_t *vp16 = vu16 + vrow;   // the four rows: immediate offsets
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
                    for (int s = 0; s < 4; ++s)
                        vr_[u][ct][s] = E::load(vp, s * d);
                }
            }
        }
    };
    // One pair of key tiles: ones column, logits, running maxima, G_U^n and T.
    auto process = [&](int t0, float (&kr)[2][8], bf8 (&kw)[2], float (&vr)[2][NCT][4],
                       uint32_t (&vh)[2][NCT][2]) {
        // The K chunks stay unmasked (their overlapping slots meet zeros in the
        // Qbar slots); V columns past d become the ones column, then zeros.
#pragma unroll
        for (int u = 0; u < 2; ++u) {
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                const int f = 16 * ct + c;
                if constexpr (BFM) {
#pragma unroll
                    for (int pp = 0; pp < 2; ++pp)
                        vh[u][ct][pp] = f < d ? vh[u][ct][pp]
                                              : (kOnes && f == d ? 0x3F803F80u : 0u);
                } else {
#pragma unroll
                    for (int s = 0; s < 4; ++s)
                        vr[u][ct][s] = f < d ? vr[u][ct][s] : (kOnes && f == d ? 1.f : 0.f);
                }
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
                    vb.w[jj] = vh[jj >> 1][ct][jj & 1];
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
                    acc = mfma_bf16(kw[u], qbh[j], acc);
                    acc = mfma_bf16(kw[u], qbl[j], acc);
                } else {
#pragma unroll
                    for (int s = 0; s < 8; ++s)
                        acc = mfma4(kr[u][s], qb[j][s], acc);
                }
                su[u] = acc;
                gmax = fmaxf(gmax, fmaxf(fmaxf(acc[0], acc[1]), fmaxf(acc[2], acc[3])));
            }
            const float mnew = fmaxf(mrun[j], max_groups(gmax));
            // Rescale what is accumulated when a maximum grew; the factor is
            // exactly 1 for every landmark whose maximum held, so skipping the
            // step when none grew changes nothing.
            if (__builtin_amdgcn_ballot_w64(mnew != mrun[j]) != 0) {
                const float f = fast_exp2(a.s2 * (mrun[j] - mnew));
                tden[j] *= f;
                const f4 fr = by_rows(f, vec, g, c);   // factor of landmark 16j + 4g + i
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
                    T[j][ct] *= fr;
            }
            mrun[j] = mnew;
            // Landmarks past m get an infinite offset: their terms are exactly 0.
            const float mb = 16 * j + c < m ? a.s2 * mnew : INFINITY;
            if constexpr (BFM) {
                float gk[8];
#pragma unroll
                for (int h = 0; h < 2; ++h)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        gk[4 * h + i] = fast_exp2(fmaf(a.s2, su[h][i], -mb));
                        if constexpr (!kOnes)
                            tden[j] += gk[4 * h + i];
                    }
                bf8 gh, gl;
                split_bf16(gk, gh, gl);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    T[j][ct] = mfma_bf16(gh, vv[ct], T[j][ct]);
                    T[j][ct] = mfma_bf16(gl, vv[ct], T[j][ct]);
                }
            } else {
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    if (u == 1 && !second)
                        break;
                    f4 e;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        e[i] = fast_exp2(fmaf(a.s2, su[u][i], -mb));
                        if constexpr (!kOnes)
                            tden[j] += e[i];
                    }
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                        for (int s = 0; s < 4; ++s)
                            T[j][ct] = mfma4(e[s], vr[u][ct][s], T[j][ct]);
                }
            }
        }
    };
    // Unrolled by two with two buffers, so that no loaded row is copied --
    // except for bf16 with three or four landmark tiles, where the unrolled
    // loop needs more registers than three waves per SIMD leave (measured
    // slower there).
    load_pair(2 * w, kr, kw, vr, vh);
    if constexpr (!(BFM && MT >= 3)) {
        for (int t0 = 2 * w; t0 < NT; t0 += 4 * kWaves) {
            load_pair(t0 + 2 * kWaves, krn, kwn, vrn, vhn);
            process(t0, kr, kw, vr, vh);
            if (t0 + 2 * kWaves >= NT)
                break;   // uniform
            load_pair(t0 + 4 * kWaves, kr, kw, vr, vh);
            process(t0 + 2 * kWaves, krn, kwn, vrn, vhn);
        }
    } else {
        for (int t0 = 2 * w; t0 < NT; t0 += 2 * kWaves) {
            load_pair(t0 + 2 * kWaves, krn, kwn, vrn, vhn);
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

    // The four waves' records, merged against the largest of their maxima.
    float *rw = recs[w];
#pragma unroll
    for (int j = 0; j < MT; ++j) {
#pragma unroll
        for (int ct = 0; ct < 2; ++ct)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float x = 0.f;
                if (ct < NCT)
                    x = T[j][ct < NCT ? ct : 0][i];
                rw[(16 * j + 4 * g + i) * kWP + 16 * ct + c] = x;
            }
        const float td = kOnes ? 0.f : sum_groups(tden[j]);
        if (g == 0) {
            rw[LD + 16 * j + c] = td;
            rw[LM + 16 * j + c] = mrun[j];
        }
    }
    __syncthreads();
    float *out = a.rec + (unit * a.nchunk + chunk) * kRec;
    for (int idx = threadIdx.x; idx < 16 * MT * (kWP / 4); idx += 64 * kWaves) {
        const int l = idx / (kWP / 4), f = 4 * (idx % (kWP / 4));
        float mx = -INFINITY;
#pragma unroll
        for (int v = 0; v < kWaves; ++v)
            mx = fmaxf(mx, recs[v][LM + l]);
        f4 acc = {0.f, 0.f, 0.f, 0.f};
        float den = 0.f;
#pragma unroll
        for (int v = 0; v < kWaves; ++v) {
            const float fw = fast_exp2(a.s2 * (recs[v][LM + l] - mx));   // 0 for an idle wave
            acc += fw * *reinterpret_cast<const f4 *>(&recs[v][l * kWP + f]);
            den += fw * recs[v][kOnes ? l * kWP + d : LD + l];
        }
        *reinterpret_cast<f4 *>(out + (f >> 2) * (kLm * 4) + 4 * l) = acc;
        if (f == 0) {
            out[kRecD + l] = den;
            out[kRecM + l] = mx;
        }
    }
}

// ---- C: merge of the chunk records ------------------------------------------
// Block (unit, landmark tile j, column group q): q < 8 merges features
// 4q .. 4q+3 of T, q = 8 the column T_D.  kMergeSlices slices of 64 threads
// take every kMergeSlices-th chunk; thread (landmark li, column x) of a slice
// keeps a running maximum and the sum against it, eight chunk records in
// flight per step (the last step's missing records read as maximum -inf,
// weight 0), and the slices are merged in LDS in a fixed order.  Every block
// of a tile computes the same maxima (a max is exact); block q = 0 stores
// s2 * m_U.
constexpr int kMergeSlices = 16;

__global__ void __launch_bounds__(64 * kMergeSlices) split_merge_kernel(SplitArgs a, int MT)
{
    constexpr int kU = 8, S = kMergeSlices;
    __shared__ float smax[S][64], ssum[S][64];
    const int per_unit = MT * kMergeGroups;
    const int64_t unit = blockIdx.x / per_unit;
    const int rem = int(blockIdx.x - unit * per_unit);
    const int j = rem / kMergeGroups, q = rem - j * kMergeGroups;
    const int slice = threadIdx.x >> 6, t = threadIdx.x & 63;
    const int li = t >> 2, x = t & 3;
    const int l = 16 * j + li;
    const int col = q < kMergeGroups - 1 ? q * (kLm * 4) + 4 * l + x : kRecD + l;   // in a record
    const int dst = q < kMergeGroups - 1 ? l * kWP + 4 * q + x : kRecD + l;         // merged
    const float *rec = a.rec + unit * a.nchunk * kRec;
    float mx = -INFINITY, sum = 0.f;
    // A step starts at a chunk below nchunk, so its maximum is finite.
    for (int ch = slice; ch < a.nchunk; ch += S * kU) {
        float cm[kU], cv[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int c = ch + S * u;
            const bool ok = c < a.nchunk;
            const float *r = rec + int64_t(ok ? c : ch) * kRec;
            const float m = r[kRecM + l], v = r[col];
            cm[u] = ok ? m : -INFINITY;
            cv[u] = ok ? v : 0.f;
        }
        float nm = mx;
#pragma unroll
        for (int u = 0; u < kU; ++u)
            nm = fmaxf(nm, cm[u]);
        sum *= fast_exp2(a.s2 * (mx - nm));   // 0 * 0 on the first step
#pragma unroll
        for (int u = 0; u < kU; ++u)
            sum = fmaf(fast_exp2(a.s2 * (cm[u] - nm)), cv[u], sum);
        mx = nm;
    }
    smax[slice][t] = mx;
    ssum[slice][t] = sum;
    __syncthreads();
    if (slice == 0) {
        float M = mx;
#pragma unroll
        for (int s = 1; s < S; ++s)
            M = fmaxf(M, smax[s][t]);
        float tot = 0.f;
#pragma unroll
        for (int s = 0; s < S; ++s)   // a slice without chunks has max -inf and weight 0
            tot += fast_exp2(a.s2 * (smax[s][t] - M)) * ssum[s][t];
        float *cb = a.comb + unit * kRec;
        cb[dst] = tot;
        if (q == 0 && x == 0)
            cb[kRecM + l] = a.s2 * M;
    }
}

// ---- P: Steps 2, 4 and 5-6 ---------------------------------------------------
template <int MT, int D, bool BFM>
__global__ void __launch_bounds__(64 * MT) split_core_kernel(SplitArgs a)
{
    using L = LargeLds<MT>;
    extern __shared__ float lds[];
    const int64_t unit = blockIdx.x;
    const int lt = wave_id(), lane = threadIdx.x & 63, g = lane >> 4, c = lane & 15;
    const int l = 16 * lt + c;
    const float *qbar = a.bar + unit * 2 * kLm * kWP, *kbar = qbar + kLm * kWP;
    const float *cb = a.comb + unit * kRec;
    for (int idx = threadIdx.x; idx < 16 * MT * kWP; idx += 64 * MT)
        lds[L::kbar + (idx / kWP) * kTS + idx % kWP] = kbar[idx];
    float qb[8];
#pragma unroll
    for (int s = 0; s < 8; ++s)
        qb[s] = slot_valid<D>(g, s) ? qbar[l * kWP + chunk_start<D>(g) + s] : 0.f;
    f4 T[2];
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
        for (int i = 0; i < 4; ++i)
            T[ct][i] = cb[(16 * lt + 4 * g + i) * kWP + 16 * ct + c];
    const float tden = cb[kRecD + l], mu = cb[kRecM + l];
    __syncthreads();   // Kbar in LDS
    landmark_core<MT, D, BFM>(lds, qb, mu, T, tden, a.m, a.iters, a.s2, lt, lane);
    float *wo = a.wout + unit * kWout;
    for (int idx = threadIdx.x; idx < table_den<MT>() + 16 * MT; idx += 64 * MT)
        wo[idx] = lds[L::wb + idx];
}

// ---- D: Steps 3 (G_L side), 6 and 7 -----------------------------------------
// With d_h % 16 != 0, column d_h of W holds Z T_D (the ones column of pass B),
// so O_D is column d_h of G_L^n W and comes out of the same products.  Each
// tile of O goes through a per-wave LDS stage and leaves as contiguous 16-byte
// pieces (O 16-byte aligned).  Landmark masks are compiled out when m fills
// its tiles.
template <bool B>
struct Flag {
    static constexpr bool value = B;
};

template <class E, int MT, int D, bool BFM>
__global__ void __launch_bounds__(64 * kWaves)
split_query_kernel(const typename E::T *__restrict__ q, typename E::T *__restrict__ o,
                   SplitArgs a)
{
    constexpr int d = D;
    constexpr bool kOnes = D % 16 != 0;
    constexpr int NCT = (D + 15) / 16;
    constexpr int TDo = table_den<MT>();
    constexpr int MP = (MT + 1) / 2;   // landmark tile pairs (bf16 path)
    constexpr int kStageBytes = 16 * D * E::bytes;   // one 16-token tile of O
    constexpr int kPieces = kStageBytes / 16;
    __shared__ __align__(16) char stages[kWaves][kStageBytes];
    __shared__ float vecs[kWaves][64];
    const int64_t unit = blockIdx.x / a.nqchunk;
    const int qc = int(blockIdx.x - unit * a.nqchunk);
    const int w = wave_id(), lane = threadIdx.x & 63, g = lane >> 4, c = lane & 15;
    float *vec = vecs[w];
    char *stage = stages[w];
    const int m = a.m;
    const int64_t base = unit * int64_t(a.N) * d;
    const typename E::T *qu = q + base;
    char *ob = reinterpret_cast<char *>(o + base);
    const float *Wb = a.wout + unit * kWout;
    const float *kbar = a.bar + unit * 2 * kLm * kWP + kLm * kWP;

    f4 WR[MT][NCT], wdv[MT];
    float kb[MT][8];
#pragma unroll
    for (int kk = 0; kk < MT; ++kk) {
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
            WR[kk][ct] = read_r<kTS>(Wb, kk, ct, g, c);
        if constexpr (!kOnes)
            wdv[kk] = *reinterpret_cast<const f4 *>(Wb + TDo + 16 * kk + 4 * g);
#pragma unroll
        for (int s = 0; s < 8; ++s)
            kb[kk][s] = slot_valid<D>(g, s) ? kbar[(16 * kk + c) * kWP + chunk_start<D>(g) + s]
                                            : 0.f;
    }
    bf8 kbh[MT], kbl[MT], wh[MP][NCT], wl[MP][NCT];
    if constexpr (BFM) {
#pragma unroll
        for (int kk = 0; kk < MT; ++kk)
            split_bf16(kb[kk], kbh[kk], kbl[kk]);
#pragma unroll
        for (int kp = 0; kp < MP; ++kp)
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
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
    const int q0 = qc * a.qchunk_len, q1 = min(a.N, q0 + a.qchunk_len);
    const int NT = (q1 - q0) >> 4;
    constexpr int kQGroup = 2;

    auto tiles = [&](auto full) {
        constexpr bool FULL = decltype(full)::value;   // m == 16 MT: no landmark masks
        // Software-pipelined as in the keys pass: the next group's Q rows are
        // requested before this group is computed.  The chunks stay unmasked:
        // the overlapping slots meet zeros on the Kbar side.
        float qg[kQGroup][8], qgn[kQGroup][8];
        bf8 qw[kQGroup], qwn[kQGroup];
        auto load_q = [&](int t0, float (&qg_)[kQGroup][8], bf8 (&qw_)[kQGroup]) {
#pragma unroll
            for (int u = 0; u < kQGroup; ++u) {
                const int64_t row = int64_t(q0 + 16 * min(t0 + u * kWaves, NT - 1) + c) * d;
                if constexpr (BFM)
                    qw_[u] = load_row8_bf16(qu16 + row + chunk_start<D>(g));
                else if constexpr (E::bytes == 4)
                    load_row8<D>(qu + row + chunk_start<D>(g), qg_[u]);
                else
                    load_chunk8<E, D>(qu + row, g, qg_[u]);
            }
        };
        load_q(w, qg, qw);
        for (int t0 = w; t0 < NT; t0 += kQGroup * kWaves) {
            load_q(t0 + kQGroup * kWaves, qgn, qwn);
#pragma unroll
            for (int u = 0; u < kQGroup; ++u) {
                const int tt = t0 + u * kWaves;
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
                        if constexpr (!kOnes)
                            od = fmaf(e, wdv[kk][i], od);
                    }
                f4 rcp;
                if constexpr (!kOnes) {
                    od = sum_groups(od);
                    const f4 odr = by_rows(od, vec, g, c);   // O_D of tokens 16tt + 4g + i
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
                f4 on[NCT];
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    f4 acc = {0.f, 0.f, 0.f, 0.f};
                    if constexpr (BFM) {
#pragma unroll
                        for (int kp = 0; kp < MP; ++kp) {
                            acc = mfma_bf16(gh[kp], wh[kp][ct], acc);
                            acc = mfma_bf16(gh[kp], wl[kp][ct], acc);
                            acc = mfma_bf16(gl[kp], wh[kp][ct], acc);
                        }
                    } else {
#pragma unroll
                        for (int kk = 0; kk < MT; ++kk)
                            acc = mm16_acc(glT[kk], WR[kk][ct], acc);
                    }
                    on[ct] = acc;
                }
                if constexpr (kOnes) {   // O_D = column d of the last feature tile
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        rcp[i] = __builtin_amdgcn_rcpf(row_bcast<D % 16>(on[NCT - 1][i]));
                }
                // The tile of O, row-major as in memory, to the stage.
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    const int f = 16 * ct + c;
                    if (f < d) {
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float x = on[ct][i] * rcp[i];
                            if constexpr (E::bytes == 4)
                                reinterpret_cast<float *>(stage)[(4 * g + i) * D + f] = x;
                            else
                                reinterpret_cast<uint16_t *>(stage)[(4 * g + i) * D + f] =
                                    uint16_t(cvt_bf16x2(x, 0.f));
                        }
                    }
                }
                wave_sync();
                f4 *dst = reinterpret_cast<f4 *>(ob + int64_t(q0 + 16 * tt) * d * E::bytes);
                const f4 *src = reinterpret_cast<const f4 *>(stage);
#pragma unroll
                for (int p0 = 0; p0 < kPieces; p0 += 64)
                    if (p0 + lane < kPieces)
                        dst[p0 + lane] = src[p0 + lane];
                wave_sync();
            }
#pragma unroll
            for (int u = 0; u < kQGroup; ++u) {
                qw[u] = qwn[u];
#pragma unroll
                for (int x = 0; x < 8; ++x)
                    qg[u][x] = qgn[u][x];
            }
        }
    };
    if (m == 16 * MT)
        tiles(Flag<true>{});
    else
        tiles(Flag<false>{});
}

// ---- host side ----------------------------------------------------------------

struct Plan {
    int pieces, piece_len, nchunk, chunk_len, nqchunk, qchunk_len;
    size_t part, bar, rec, comb, wout, bytes;   // byte offsets of the regions, total
};

constexpr int64_t kTargetBlocks = 2048;   // workgroups per streaming pass (8 per CU)

int64_t ceil_div(int64_t x, int64_t y) { return (x + y - 1) / y; }
int64_t round_up(int64_t x, int64_t y) { return ceil_div(x, y) * y; }

// Chunk length for a streaming pass: enough chunks for kTargetBlocks
// workgroups over all units, at least `lo` and at most `hi` tokens, a
// multiple of `mult`.
int chunk_length(int64_t units, int N, int mult, int lo, int hi)
{
    const int64_t per_unit = ceil_div(kTargetBlocks, units);
    int64_t len = round_up(ceil_div(N, per_unit), mult);
    len = len < lo ? lo : (len > hi ? hi : len);
    const int64_t whole = round_up(N, mult);
    return int(len < whole ? len : whole);
}

Plan make_plan(const Problem &p)
{
    Plan s;
    const int P = p.geo.pr * p.geo.pc;
    const int64_t units = p.units > 0 ? p.units : 1;
    int pieces = int(ceil_div(kTargetBlocks, units * p.m));
    const int most = P / 64 > 1 ? P / 64 : 1;   // pieces of at least 64 tokens
    pieces = pieces < 1 ? 1 : (pieces > most ? most : pieces);
    s.piece_len = int(ceil_div(P, pieces));
    s.pieces = int(ceil_div(P, s.piece_len));
    s.chunk_len = chunk_length(units, p.N, 32, 256, 4096);
    s.nchunk = int(ceil_div(p.N, s.chunk_len));
    s.qchunk_len = chunk_length(units, p.N, 16 * kWaves * 2, 256, 4096);
    s.nqchunk = int(ceil_div(p.N, s.qchunk_len));
    size_t off = 0;
    auto region = [&](size_t floats) {
        const size_t at = off;
        off += round_up(int64_t(floats * sizeof(float)), 256);
        return at;
    };
    const size_t u = size_t(units);
    s.part = region(u * 2 * size_t(p.m) * s.pieces * kWP);
    s.bar = region(u * 2 * kLm * kWP);
    s.rec = region(u * size_t(s.nchunk) * kRec);
    s.comb = region(u * kRec);
    s.wout = region(u * kWout);
    s.bytes = off;
    return s;
}

template <class E, int MT, int D>
void launch_split_md(const Problem &p, const Plan &s, const SplitArgs &a, hipStream_t stream)
{
    const auto *q = static_cast<const typename E::T *>(p.q);
    const auto *k = static_cast<const typename E::T *>(p.k);
    const auto *v = static_cast<const typename E::T *>(p.v);
    auto *o = static_cast<typename E::T *>(p.o);
    const unsigned U = unsigned(p.units);
    const dim3 block(64 * kWaves);
    hipLaunchKernelGGL((split_pool_kernel<E, D>), dim3(U * unsigned(p.m * s.pieces)), block, 0,
                       stream, q, k, a);
    hipLaunchKernelGGL(split_bar_kernel, dim3(U * 2 * kLm), dim3(64), 0, stream, a);
    const bool bfm = E::bytes == 2 && p.N % 32 == 0;
    if (bfm)
        hipLaunchKernelGGL((split_keys_kernel<E, MT, D, E::bytes == 2>),
                           dim3(U * unsigned(s.nchunk)), block, 0, stream, k, v, a);
    else
        hipLaunchKernelGGL((split_keys_kernel<E, MT, D, false>), dim3(U * unsigned(s.nchunk)),
                           block, 0, stream, k, v, a);
    hipLaunchKernelGGL(split_merge_kernel, dim3(U * unsigned(MT * kMergeGroups)),
                       dim3(64 * kMergeSlices), 0, stream, a, MT);
    const size_t lds = size_t(LargeLds<MT>::total) * sizeof(float);
    if (bfm)
        hipLaunchKernelGGL((split_core_kernel<MT, D, E::bytes == 2>), dim3(U), dim3(64 * MT), lds,
                           stream, a);
    else
        hipLaunchKernelGGL((split_core_kernel<MT, D, false>), dim3(U), dim3(64 * MT), lds, stream,
                           a);
    if (bfm)
        hipLaunchKernelGGL((split_query_kernel<E, MT, D, E::bytes == 2>),
                           dim3(U * unsigned(s.nqchunk)), block, 0, stream, q, o, a);
    else
        hipLaunchKernelGGL((split_query_kernel<E, MT, D, false>), dim3(U * unsigned(s.nqchunk)),
                           block, 0, stream, q, o, a);
}

template <class E, int D>
void launch_split_d(const Problem &p, const Plan &s, const SplitArgs &a, hipStream_t stream)
{
    switch ((p.m + 15) / 16) {
    case 1: launch_split_md<E, 1, D>(p, s, a, stream); break;
    case 2: launch_split_md<E, 2, D>(p, s, a, stream); break;
    case 3: launch_split_md<E, 3, D>(p, s, a, stream); break;
    default: launch_split_md<E, 4, D>(p, s, a, stream); break;
    }
}

template <class E>
void launch_split_e(const Problem &p, const Plan &s, const SplitArgs &a, hipStream_t stream)
{
    switch (p.d) {
    case 8: launch_split_d<E, 8>(p, s, a, stream); break;
    case 12: launch_split_d<E, 12>(p, s, a, stream); break;
    case 16: launch_split_d<E, 16>(p, s, a, stream); break;
    case 20: launch_split_d<E, 20>(p, s, a, stream); break;
    case 24: launch_split_d<E, 24>(p, s, a, stream); break;
    case 28: launch_split_d<E, 28>(p, s, a, stream); break;
    case 30: launch_split_d<E, 30>(p, s, a, stream); break;
    default: launch_split_d<E, 32>(p, s, a, stream); break;
    }
}

}  // namespace

bool split_supported(const Problem &p)
{
    if (p.N % 16 != 0 || p.m > 64 || !tiled_width(p.d) || uintptr_t(p.o) % 16 != 0)
        return false;
    if (p.dtype == 1) {   // 16-byte row pieces of bf16 need 4-byte aligned rows
        const uintptr_t mis = uintptr_t(p.q) | uintptr_t(p.k) | uintptr_t(p.v);
        if (mis % 4 != 0)
            return false;
    }
    // every grid within the 2^32 work-items of one dispatch dimension
    const Plan s = make_plan(p);
    int64_t most = s.nchunk > s.nqchunk ? s.nchunk : s.nqchunk;
    if (int64_t(p.m) * s.pieces > most)
        most = int64_t(p.m) * s.pieces;
    if (most < 4 * kMergeGroups)
        most = 4 * kMergeGroups;
    return p.units * most * 256 < (int64_t(1) << 32);
}

size_t split_workspace_bytes(const Problem &p) { return make_plan(p).bytes; }

hipError_t launch_split(const Problem &p, void *workspace, hipStream_t stream)
{
    const Plan s = make_plan(p);
    char *ws = static_cast<char *>(workspace);
    SplitArgs a;
    a.units = p.units;
    a.N = p.N;
    a.d = p.d;
    a.m = p.m;
    a.iters = p.iters;
    a.s2 = p.scale * kLog2e;
    a.P = p.geo.pr * p.geo.pc;
    a.inv_patch = 1.0f / float(a.P);
    a.cols = p.geo.cols;
    a.pr = p.geo.pr;
    a.pc = p.geo.pc;
    a.gc = p.geo.gc;
    a.pieces = s.pieces;
    a.piece_len = s.piece_len;
    a.nchunk = s.nchunk;
    a.chunk_len = s.chunk_len;
    a.nqchunk = s.nqchunk;
    a.qchunk_len = s.qchunk_len;
    a.part = reinterpret_cast<float *>(ws + s.part);
    a.bar = reinterpret_cast<float *>(ws + s.bar);
    a.rec = reinterpret_cast<float *>(ws + s.rec);
    a.comb = reinterpret_cast<float *>(ws + s.comb);
    a.wout = reinterpret_cast<float *>(ws + s.wout);
    if (p.dtype == 0)
        launch_split_e<F32>(p, s, a, stream);
    else
        launch_split_e<BF16>(p, s, a, stream);
    return hipGetLastError();
}

}  // namespace nystra
