// Landmark-side core of the MFMA-tiled Nystrom kernels: Step 2 (G_A^n),
// Step 4 (the pseudo-inverse iteration) and Steps 5-6 re-associated
// (W = Z T, W_D = Z T_D), for one (window, head) unit whose MT landmark tiles
// are owned one per wavefront of the workgroup.
//
// Matrices shared between waves sit in LDS row-major with a padded pitch: a
// right-hand operand tile is read as four strided words per lane, the
// transpose of an own-row tile as one 16-byte word per lane.
#pragma once

#include "tile_common.hpp"

namespace nystra {
namespace core {

using namespace tile;

constexpr int kTS = 36;   // pitch of [landmark][feature] tables (Kbar, T, W)


// LDS carve-up (floats) for MT landmark tiles.
template <int MT>
struct LargeLds {
    static constexpr int M = 16 * MT;
    static constexpr int P = M + 4;    // pitch (floats) of fp32 m x m matrices
    // Pitch (bf16 elements) of the transposed bf16 matrices.  Rows 2 words
    // (mod 4) apart keep the 8-byte operand reads of 16 lanes on distinct
    // banks (a pitch of 4 words mod 8 puts lanes c and c + 8 of a row group
    // on one bank pair: measured a third slower).  One landmark tile keeps
    // M + 8, which the key-pass records need.
    static constexpr int PB = MT == 1 ? M + 8 : M + 4;
    static constexpr int RS = M * PB;  // one matrix region (floats): fp32 [M][P] or bf16 hi+lo
    static constexpr int kbar = 0;
    static constexpr int zb = kbar + M * kTS;
    static constexpr int ya = zb + RS;
    static constexpr int yb = ya + RS;                  // also the own-row transpose scratch
    static constexpr int vec = yb + RS;                 // [MT][64] row vectors
    // Z_0's column-sum partials [MT][M] and row-sum maxima [MT] (padded) share
    // the row-vector region, which no wave uses between the key pass and the
    // query pass.
    static constexpr int vec_len = 64 * MT > MT * M + 4 ? 64 * MT : MT * M + 4;
    static constexpr int colpart = vec;
    static constexpr int rowmax = colpart + MT * M;
    // Before the landmark core runs, its matrix regions hold the key pass of
    // the one-pass large kernel: the Qbar table and one record per wave (T
    // rows of every landmark, pitch kRecP; T_D; running maxima).
    static constexpr int kRecP = 32;
    static constexpr int rec_len = M * kRecP + 2 * M;
    static constexpr int qtab = zb;
    static constexpr int recs = qtab + M * kTS;
    // After the iteration the T table starts at zb and the W table ends at
    // vec (both may run into the dead middle region); otherwise they follow.
    static constexpr int tab_len = M * kTS + M;         // table + its denominator column
    static constexpr bool tab_in = 2 * tab_len <= 3 * RS;
    static constexpr int tb = tab_in ? zb : vec + vec_len;
    static constexpr int wb = tab_in ? vec - tab_len : tb + tab_len;
    static constexpr int total = tab_in ? vec + vec_len : wb + tab_len;
    static_assert(recs + MT * rec_len <= vec, "key-pass records fit the matrix regions");
    static_assert((M - 1) * P + M <= RS, "the fp32 scratch fits its region");
    static_assert(tb + tab_len <= wb, "the T and W tables do not overlap");
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

// bf16 copies of an m x m matrix for the bf16 matrix cores: hi and lo terms,
// each stored transposed ([column][row], pitch PB) so that the right-hand
// operand of a 32-deep product -- rows 32kp + 4g .. +3 and 32kp + 16 + 4g .. +3
// of one column -- is two 8-byte reads.  The writer splits once.
template <int M, int PB>
__device__ inline void publish_bf(uint16_t *reg, int a, int b, f4 v, int g, int c)
{
    // Pairs converted together (round to nearest even): the values of an
    // element-wise split.
    const NegSel s = neg_selectors();
    uint32_t h[2], l[2];
#pragma unroll
    for (int p = 0; p < 2; ++p) {
        h[p] = cvt_bf16x2(v[2 * p], v[2 * p + 1]);
        l[p] = residual_bf16x2(h[p], v[2 * p], v[2 * p + 1], s);
    }
    uint16_t *hp = reg + (16 * b + c) * PB + 16 * a + 4 * g;
    *reinterpret_cast<uint2 *>(hp) = make_uint2(h[0], h[1]);
    *reinterpret_cast<uint2 *>(hp + M * PB) = make_uint2(l[0], l[1]);
}

template <int M, int PB>
__device__ inline void read_pair_bf(const uint16_t *reg, int kp, int j, int g, int c, bf8 &bh,
                                    bf8 &bl)
{
    const uint16_t *p = reg + (16 * j + c) * PB + 32 * kp + 4 * g;
    const uint2 a0 = *reinterpret_cast<const uint2 *>(p);
    const uint2 a1 = *reinterpret_cast<const uint2 *>(p + 16);
    const uint2 b0 = *reinterpret_cast<const uint2 *>(p + M * PB);
    const uint2 b1 = *reinterpret_cast<const uint2 *>(p + M * PB + 16);
    U16B h, l;
    h.w[0] = a0.x; h.w[1] = a0.y; h.w[2] = a1.x; h.w[3] = a1.y;
    l.w[0] = b0.x; l.w[1] = b0.y; l.w[2] = b1.x; l.w[3] = b1.y;
    bh = __builtin_bit_cast(bf8, h);
    bl = __builtin_bit_cast(bf8, l);
}

// Left operand of a 32-deep product from two transposed row tiles.
__device__ inline void split_pair(f4 t0, f4 t1, bf8 &hi, bf8 &lo)
{
    float x[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[i] = t0[i];
        x[4 + i] = t1[i];
    }
    split_bf16(x, hi, lo);
}

// Offset (floats) of the denominator column in a [landmark][feature] table.
template <int MT>
constexpr int table_den() { return 16 * MT * kTS; }

// Steps 2, 4 and 5-6 for the unit held by this workgroup; wave lt owns
// landmark tile lt and lane (g, c) the landmark l = 16 lt + c.
//   qb    this lane's eight feature slots of Qbar row l (load_chunk8 layout)
//   mu    s2 * m_U of landmark l (the row maximum of S_U, base-2 units)
//   T     this wave's rows of T = G_U^n V in D-layout, feature tiles 0 and 1
//   tden  T_D of landmark l (sum of row l of G_U^n)
// Kbar must be complete in LDS (LargeLds::kbar, pitch kTS) and visible to all
// waves.  On return, after a workgroup barrier, W and W_D are in the table at
// LargeLds::wb (W_D at offset table_den<MT>()).  FULL says m = 16 MT (every
// landmark slot real), which folds the masks.
template <int MT, int D, bool BFM, bool FULL = false>
__device__ inline void landmark_core(float *lds, const float (&qb)[8], float mu,
                                              const f4 (&T)[2], float tden, int m, int iters,
                                              float s2, int lt, int lane)
{
    using L = LargeLds<MT>;
    constexpr int M = L::M, P = L::P;
    float *kbar = lds + L::kbar, *colpart = lds + L::colpart;
    float *rowmax = lds + L::rowmax, *Zb = lds + L::zb, *Ya = lds + L::ya, *Yb = lds + L::yb;
    float *Tb = lds + L::tb, *Wb = lds + L::wb;
    const int g = lane >> 4, c = lane & 15;
    const int l = 16 * lt + c;
    const bool lval = FULL || l < m;

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
            ALT[j][i] = (lval && (FULL || 16 * j + 4 * g + i < m))
                            ? fast_exp2(fmaf(s2, acc[i], -mu)) : 0.f;
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
    f4 eye;   // identity of the m x m block on this wave's diagonal tile
#pragma unroll
    for (int i = 0; i < 4; ++i)
        eye[i] = (4 * g + i == c && lval) ? 1.f : 0.f;
    const f4 zero4 = {0.f, 0.f, 0.f, 0.f};
    f4 ZLT[MT];   // ZLT[j] lane (g,c): Z[16lt + c][16j + 4g + i]

    // bf16 inputs with an even number of landmark tiles run the iteration on the
    // bf16 matrix cores, every operand carried as hi + lo terms (three products).
    constexpr bool BFP = BFM && (MT % 2 == 0);
    if constexpr (BFP) {
        constexpr int MP = MT / 2, PB = L::PB;
        uint16_t *Zh = reinterpret_cast<uint16_t *>(Zb), *Yah = reinterpret_cast<uint16_t *>(Ya);
        uint16_t *Ybh = reinterpret_cast<uint16_t *>(Yb);
        float *scr = Yb;   // fp32 own-row transposes (rows 16lt .. 16lt+15)
        // Z_0 = alpha A^T: bf16 copies for the products, an fp32 copy in scr for
        // this wave's own row.
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            publish_bf<M, PB>(Zh, j, lt, ALT[j] * alpha, g, c);
            write_tile<P>(scr, j, lt, ALT[j] * alpha, g, c);
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < MT; ++j)
            ZLT[j] = read_lt<P>(scr, lt, j, g, c);
        bf8 ah[MP], al[MP];
#pragma unroll
        for (int kp = 0; kp < MP; ++kp)
            split_pair(ALT[2 * kp], ALT[2 * kp + 1], ah[kp], al[kp]);
        auto product = [&](const bf8 *lh, const bf8 *ll, const uint16_t *reg, int j) {
            f4 acc = zero4;
#pragma unroll
            for (int kp = 0; kp < MP; ++kp) {
                bf8 bh, bl;
                read_pair_bf<M, PB>(reg, kp, j, g, c, bh, bl);
                acc = mfma_bf16(lh[kp], bh, acc);
                acc = mfma_bf16(lh[kp], bl, acc);
                acc = mfma_bf16(ll[kp], bh, acc);
            }
            return acc;
        };
        __syncthreads();   // every wave has read its Z_0 row before scr is reused
        for (int it = 0; it < iters; ++it) {
            f4 X[MT];
#pragma unroll
            for (int j = 0; j < MT; ++j)
                X[j] = product(ah, al, Zh, j);
#pragma unroll
            for (int j = 0; j < MT; ++j)
                write_tile<P>(scr, lt, j, X[j], g, c);
            wave_sync();
            bf8 xh[MP], xl[MP];
#pragma unroll
            for (int kp = 0; kp < MP; ++kp)
                split_pair(read_lt<P>(scr, lt, 2 * kp, g, c), read_lt<P>(scr, lt, 2 * kp + 1, g, c),
                           xh[kp], xl[kp]);
#pragma unroll
            for (int j = 0; j < MT; ++j)
                publish_bf<M, PB>(Yah, lt, j, (j == lt ? eye * 7.f : zero4) - X[j], g, c);
            __syncthreads();
            f4 Y[MT];
#pragma unroll
            for (int j = 0; j < MT; ++j)
                Y[j] = (j == lt ? eye * 15.f : zero4) - product(xh, xl, Yah, j);
#pragma unroll
            for (int j = 0; j < MT; ++j)
                publish_bf<M, PB>(Ybh, lt, j, Y[j], g, c);
            __syncthreads();
#pragma unroll
            for (int j = 0; j < MT; ++j)
                Y[j] = (j == lt ? eye * 13.f : zero4) - product(xh, xl, Ybh, j);
#pragma unroll
            for (int j = 0; j < MT; ++j)
                publish_bf<M, PB>(Yah, lt, j, Y[j], g, c);
            __syncthreads();
            bf8 zh[MP], zl[MP];
#pragma unroll
            for (int kp = 0; kp < MP; ++kp)
                split_pair(ZLT[2 * kp], ZLT[2 * kp + 1], zh[kp], zl[kp]);
            f4 Zn[MT];
#pragma unroll
            for (int j = 0; j < MT; ++j)
                Zn[j] = product(zh, zl, Yah, j) * 0.25f;
#pragma unroll
            for (int j = 0; j < MT; ++j) {
                publish_bf<M, PB>(Zh, lt, j, Zn[j], g, c);
                write_tile<P>(scr, lt, j, Zn[j], g, c);
            }
            wave_sync();
#pragma unroll
            for (int j = 0; j < MT; ++j)
                ZLT[j] = read_lt<P>(scr, lt, j, g, c);
            __syncthreads();
        }
    } else {
    // Z_0[j][lt] = alpha (A[lt][j])^T, whose D-layout is alpha * ALT[j].
#pragma unroll
    for (int j = 0; j < MT; ++j)
        write_tile<P>(Zb, j, lt, ALT[j] * alpha, g, c);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < MT; ++j)
        ZLT[j] = read_lt<P>(Zb, lt, j, g, c);
    __syncthreads();   // every wave has its Z_0 row (the T table may follow in Zb)

    // Iteration: X = A Z; Z <- Z (13I - X (15I - X (7I - X))) / 4, each wave
    // producing its row tile of every product.
    for (int it = 0; it < iters; ++it) {
        f4 X[MT];
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            f4 acc = zero4;
#pragma unroll
            for (int kk = 0; kk < MT; ++kk)
                acc = mm16_acc(ALT[kk], read_r<P>(Zb, kk, j, g, c), acc);
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
            write_tile<P>(Ya, lt, j, X[j], g, c);
        __syncthreads();
        // The update in expanded form, the constants riding in the products'
        // accumulators: Y1 = 15I - 7X + X X, N = X Y1 - 13I (= -Y2) and
        // Z <- -(Z N) / 4.
        f4 Y[MT];
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            f4 acc;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                acc[i] = fmaf(X[j][i], -7.f, j == lt ? 15.f * eye[i] : 0.f);
#pragma unroll
            for (int kk = 0; kk < MT; ++kk)
                acc = mm16_acc(XLT[kk], read_r<P>(Ya, kk, j, g, c), acc);
            Y[j] = acc;
        }
#pragma unroll
        for (int j = 0; j < MT; ++j)
            write_tile<P>(Yb, lt, j, Y[j], g, c);
        __syncthreads();
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            f4 acc = j == lt ? eye * -13.f : zero4;
#pragma unroll
            for (int kk = 0; kk < MT; ++kk)
                acc = mm16_acc(XLT[kk], read_r<P>(Yb, kk, j, g, c), acc);
            Y[j] = acc;
        }
#pragma unroll
        for (int j = 0; j < MT; ++j)
            write_tile<P>(Ya, lt, j, Y[j], g, c);
        __syncthreads();
        f4 Zn[MT];
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            f4 acc = zero4;
#pragma unroll
            for (int kk = 0; kk < MT; ++kk)
                acc = mm16_acc(ZLT[kk], read_r<P>(Ya, kk, j, g, c), acc);
            Zn[j] = acc * -0.25f;
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
    }

    // ---- Steps 5-6 re-associated: W = Z T and W_D = Z T_D.
    constexpr int TDo = table_den<MT>();
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
            acc = mm16_acc(ZLT[kk], read_r<kTS>(Tb, kk, ct, g, c), acc);
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
}

}  // namespace core
}  // namespace nystra
