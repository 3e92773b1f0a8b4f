// MFMA-tiled PnP-Nystra kernel for small windows (N = 16, 32 or 64 tokens,
// m <= 16 landmarks, d_h in {8, 12, ..., 28, 30, 32}): one wavefront computes one
// (window, head) unit in registers (register tiles in the D-layout of
// tile_common.hpp), with LDS holding the pooling exchange and small
// transposes.  fp32 inputs
// run every contraction on v_mfma_f32_16x16x4f32; bf16 inputs run the
// products with Q, K and V on v_mfma_f32_16x16x32_bf16, the fp32 partner
// operand split into bf16 hi + lo terms, run the pseudo-inverse products as
// (hi + lo) x (hi + lo) bf16 terms, and keep S_A and W = Z T in fp32.
//
// Contractions over the feature dimension (S_L, S_U, S_A) use eight MFMA
// steps in which each lane group supplies a chunk of 8 consecutive features
// of one token row, loaded straight from global memory in 16-byte pieces.
// The last group's chunk is shifted back to end at the row end, so it
// overlaps the group below; the overlap is zeroed on the landmark side, and
// all global loads are branch-free and in bounds.  When d_h leaves a spare
// column in the last 16-wide feature tile, that column of V is replaced by
// ones, so the value products also carry the denominators T_D, W_D and O_D.
#include "internal.hpp"
#include "tile_common.hpp"

namespace nystra {
namespace {

using namespace tile;

constexpr int kWavesPerBlock = 4;

// Pooling grids of the 8x8 windows that restoration models use, fixed at
// compile time: kGrid2x2 is m = 16 (4 x 4 patches of 2 x 2 tokens), kGrid2x4
// is m = 8 (4 x 2 patches of 2 rows x 4 columns).  kGridAny reads the grid
// from SmallArgs.
enum { kGridAny = 0, kGrid2x2 = 1, kGrid2x4 = 2 };

// Row stride (floats) of the raw Q / K chunks staged for the fixed grids: a
// token's four 8-feature chunks plus 16 bytes of padding.
template <class E>
constexpr int raw_stride() { return E::bytes == 4 ? 36 : 20; }

// LDS of one wave: the landmark rows of Q and K (slot layout; with a fixed
// grid, the staged raw chunks of one input instead), the transpose scratch of
// the pseudo-inverse and a row vector.  V and O move between registers and
// HBM directly.
template <class E, int NT, int D, int GRID>
struct SmallLds {
    static constexpr int kRows =
        GRID == kGridAny ? 2 * 16 * kLdStride : 16 * NT * raw_stride<E>();
    static constexpr int kStage = 16 * kTrStride;
    static constexpr int kPerWave = kRows + kStage + 64;
};

struct SmallArgs {
    int64_t units;
    int m, iters;
    float s2;          // logit scale in base-2 units (scale * log2 e)
    float inv_patch;   // 1 / tokens per pooling patch (a power of two)
    int lg_cols, lg_pr, lg_pc, lg_gc, free_bits;   // pooling grid (log2 sizes)
};

int grid_of(const SmallArgs &a, int N)
{
    if (N == 64 && a.m == 16 && a.lg_cols == 3 && a.lg_pr == 1 && a.lg_pc == 1 && a.lg_gc == 2 &&
        a.free_bits == 9)
        return kGrid2x2;
    if (N == 64 && a.m == 8 && a.lg_cols == 3 && a.lg_pr == 1 && a.lg_pc == 2 && a.lg_gc == 1 &&
        a.free_bits == 11)
        return kGrid2x4;
    return kGridAny;
}

// Step 1 for one input: the patch sums of this wave's tokens (the mean times
// the patch size; the factor is folded into the logit scales, exactly, since
// the patch size is a power of two), written to bar[l][8g + s] in the slot
// layout of the feature chunks with the overlapping slots zeroed.  A patch is
// the set of tokens that agree with its base token outside the bit mask
// `free_bits`: tile bits are summed within the lane (base tiles only), lane
// bits across lanes by DPP / swizzle exchanges.  get(tt, x) yields the eight
// chunk values of tile tt.
template <int NT, int D, class Get>
__device__ inline void pool_to_lds(Get get, float *bar, const SmallArgs &a, int g, int c)
{
    const int lane_bits = a.free_bits & 15, tile_bits = a.free_bits >> 4;
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
        if (tt & tile_bits)
            continue;   // uniform: only base tiles of a patch produce a sum
        float acc[8];
        get(tt, acc);
#pragma unroll
        for (int u = 0; u < NT; ++u)
            if (u != tt && ((u ^ tt) & ~tile_bits) == 0) {
                float y[8];
                get(u, y);
#pragma unroll
                for (int s = 0; s < 8; ++s)
                    acc[s] += y[s];
            }
        if (lane_bits & 1)
#pragma unroll
            for (int s = 0; s < 8; ++s)
                acc[s] += dpp_xor1(acc[s]);
        if (lane_bits & 2)
#pragma unroll
            for (int s = 0; s < 8; ++s)
                acc[s] += dpp_xor2(acc[s]);
        if (lane_bits & 4)
#pragma unroll
            for (int s = 0; s < 8; ++s)
                acc[s] += swz_xor4(acc[s]);
        if (lane_bits & 8)
#pragma unroll
            for (int s = 0; s < 8; ++s)
                acc[s] += dpp_xor8(acc[s]);
#pragma unroll
        for (int s = 0; s < 8; ++s)
            acc[s] = slot_keep<D>(g, s) ? acc[s] : 0.f;
        // The exchanges are butterflies of commutative additions, so every
        // lane of a patch holds the same sum bit for bit: all of them store
        // it (no branch), each to its own token's landmark row.
        const int t = 16 * tt + c;
        const int r = t >> a.lg_cols, cc = t & ((1 << a.lg_cols) - 1);
        const int l = ((r >> a.lg_pr) << a.lg_gc) + (cc >> a.lg_pc);
        f4 *dst = reinterpret_cast<f4 *>(bar + l * kLdStride + 8 * g);
        dst[0] = f4{acc[0], acc[1], acc[2], acc[3]};
        dst[1] = f4{acc[4], acc[5], acc[6], acc[7]};
    }
}

// Stages the raw chunk of token tile tt (this lane's token 16tt + c, feature
// group g) in the LDS row of its token.
template <class E, class Chunk>
__device__ inline void stage_chunk(const Chunk &x, float *stage, int tt, int g, int c)
{
    constexpr int RS = raw_stride<E>();
    float *row = stage + (16 * tt + c) * RS + (E::bytes == 4 ? 8 : 4) * g;
    if constexpr (E::bytes == 4) {
        reinterpret_cast<f4 *>(row)[0] = f4{x[0], x[1], x[2], x[3]};
        reinterpret_cast<f4 *>(row)[1] = f4{x[4], x[5], x[6], x[7]};
    } else {
        *reinterpret_cast<U16B *>(row) = __builtin_bit_cast(U16B, x);
    }
}

// Lane (g, c) adds the staged chunks of the tokens of landmark c's patch, in
// patch order: out[s] = patch sum of slot s of group g (zero in overlapping
// slots and for padding landmarks).
template <class E, int D, int GRID>
__device__ inline void patch_sums(const float *stage, float (&out)[8], int m, int g, int c)
{
    constexpr int RS = raw_stride<E>();
    constexpr int PR = 2, PC = GRID == kGrid2x2 ? 2 : 4, GC = 8 / PC;   // 8 x 8 window
    const int le = min(c, m - 1);   // padding lanes read a valid patch, then drop it
    const int r0 = (le / GC) * PR, c0 = (le % GC) * PC;
#pragma unroll
    for (int s = 0; s < 8; ++s)
        out[s] = 0.f;
#pragma unroll
    for (int i = 0; i < PR; ++i)
#pragma unroll
        for (int j = 0; j < PC; ++j) {
            const float *row = stage + ((r0 + i) * 8 + c0 + j) * RS + (E::bytes == 4 ? 8 : 4) * g;
            if constexpr (E::bytes == 4) {
                const f4 a = reinterpret_cast<const f4 *>(row)[0];
                const f4 b = reinterpret_cast<const f4 *>(row)[1];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    out[u] += a[u];
                    out[4 + u] += b[u];
                }
            } else {
                const U16B w = *reinterpret_cast<const U16B *>(row);
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    out[2 * u] += __uint_as_float(w.w[u] << 16);
                    out[2 * u + 1] += __uint_as_float(w.w[u] & 0xffff0000u);
                }
            }
        }
    const bool valid = c < m;
#pragma unroll
    for (int s = 0; s < 8; ++s)
        out[s] = (valid && slot_keep<D>(g, s)) ? out[s] : 0.f;
}

// Step 1 for a fixed grid, one input, all NT token tiles held by one wave:
// stage every chunk, then form the patch sums.
template <class E, int NT, int D, int GRID, class Chunk>
__device__ inline void pool_direct(const Chunk (&x)[NT], float *stage, float (&out)[8], int m,
                                   int g, int c)
{
#pragma unroll
    for (int tt = 0; tt < NT; ++tt)
        stage_chunk<E>(x[tt], stage, tt, g, c);
    wave_sync();
    patch_sums<E, D, GRID>(stage, out, m, g, c);
    wave_sync();
}

__device__ inline uint32_t pack_bf16x2(float lo, float hi)
{
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2{lo, hi}), b2));   // RNE
}

// Resident waves per SIMD are capped below what the registers allow (three
// for fp32, four for bf16): with fewer waves resident than units per SIMD,
// the waves that start later load their inputs while the first ones
// compute.  With every unit resident at once (the SwinIR-like layer has six
// per SIMD) all loads are issued at the start and all computation follows.
// On that layer the caps measured fastest (fp32 47.2 -> 45.1 us at three
// waves instead of four, bf16 33.8 -> 29.9 us at four instead of six); on
// L2-resident inputs the computation alone runs at the same speed from three
// to six waves.
// KF > 0 fixes the number of pseudo-inverse iterations at compile time (the
// loop is unrolled); KF = 0 takes it from SmallArgs.
template <class E, int NT, int D, bool BFM, int GRID, int KF>
__global__ void __launch_bounds__(64 * kWavesPerBlock)
__attribute__((amdgpu_waves_per_eu(1, BFM ? 4 : 3)))
tiled_small_kernel(const typename E::T *__restrict__ q, const typename E::T *__restrict__ k,
                   const typename E::T *__restrict__ v, typename E::T *__restrict__ o,
                   SmallArgs a)
{
    constexpr int N = 16 * NT;
    constexpr int NCT = (D + 15) / 16;   // 16-wide feature tiles of V, T, W and O
    // With a spare feature column (D not a multiple of 16), column D of V is
    // replaced by ones, so that column D of T, W and O carries T_D, W_D, O_D.
    constexpr bool PAD = D % 16 != 0;
    using L = SmallLds<E, NT, D, GRID>;
    // L::kPerWave floats per wave of the workgroup (sized at launch)
    extern __shared__ __attribute__((aligned(16))) float lds_all[];
    // The wave index is uniform across the wavefront; saying so keeps the
    // unit's base addresses in scalar registers.
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int g = lane >> 4, c = lane & 15;
    const int64_t unit = int64_t(blockIdx.x) * (blockDim.x >> 6) + wave;
    if (unit >= a.units)
        return;   // whole wavefront; the kernel has no block-level barrier
    // The fixed grids imply m (16 for 2 x 2 patches, 8 for 2 x 4), so the
    // landmark masks fold away.
    const int m = GRID == kGrid2x2 ? 16 : GRID == kGrid2x4 ? 8 : a.m;
    float *qbar = lds_all + wave * L::kPerWave;
    float *kbar = qbar + 16 * kLdStride;
    float *scr = qbar + L::kRows;   // transpose scratch
    float *vec = scr + L::kStage;

    const int64_t base = unit * int64_t(N) * D;
    const typename E::T *qu = q + base, *ku = k + base, *vu = v + base;
    typename E::T *ou = o + base;

    // ---- Step 1 loads: chunk (features f0(g).., token 16tt+c) of Q and K;
    // bf16 inputs keep their raw bits for the bf16 matrix cores.
    const int f0 = chunk_start<D>(g);
    float qr[NT][8], kr[NT][8];
    bf8 qw[NT], kw[NT];
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
        const int off = (16 * tt + c) * D + f0;
        if constexpr (BFM) {
            qw[tt] = load_row8_bf16(reinterpret_cast<const uint16_t *>(qu) + off);
            kw[tt] = load_row8_bf16(reinterpret_cast<const uint16_t *>(ku) + off);
        } else {
            load_row8<D>(qu + off, qr[tt]);
            load_row8<D>(ku + off, kr[tt]);
        }
    }
    // V in the right-hand operand layout of T = G_U^n V, loaded from HBM
    // together with Q and K, so that a unit's three blocks arrive together:
    // vr[tt][ct][s] = V[token 16tt+4g+s][feature 16ct+c].  Columns past D read
    // column D-1 and never reach a stored output; column D becomes the ones
    // column.
    float vr[NT][NCT][4];
    uint16_t vh[NT][NCT][4];
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) {
        const int f = 16 * ct + c;
        const int vlane = 4 * g * D + min(f, D - 1);
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int idx = vlane + (16 * tt + s) * D;
                const bool ones = PAD && ct == NCT - 1 && f == D;
                if constexpr (BFM) {
                    const uint16_t x = reinterpret_cast<const uint16_t *>(vu)[idx];
                    vh[tt][ct][s] = ones ? uint16_t(0x3F80) : x;   // bf16 1.0
                } else {
                    const float x = E::load(vu, idx);
                    vr[tt][ct][s] = ones ? 1.f : x;
                }
            }
    }

    __builtin_amdgcn_sched_barrier(0);

    // Landmark rows in slot layout: kb[s] = Kbar[c][slot s of group g] (zero
    // in overlapping slots), qb likewise (patch sums).
    float kb[8], qb[8];
    if constexpr (GRID != kGridAny) {
        if constexpr (BFM) {
            pool_direct<E, NT, D, GRID>(qw, qbar, qb, m, g, c);
            pool_direct<E, NT, D, GRID>(kw, qbar, kb, m, g, c);
        } else {
            pool_direct<E, NT, D, GRID>(qr, qbar, qb, m, g, c);
            pool_direct<E, NT, D, GRID>(kr, qbar, kb, m, g, c);
        }
    } else {
        // Landmark rows m..15 are padding: zero them so they contribute nothing.
        for (int idx = lane; idx < (16 - m) * 32; idx += 64) {
            const int r = m + idx / 32, f = idx % 32;
            qbar[r * kLdStride + f] = 0.f;
            kbar[r * kLdStride + f] = 0.f;
        }
        if constexpr (BFM) {
            pool_to_lds<NT, D>([&](int tt, float *x) { unpack_bf8(qw[tt], x); }, qbar, a, g, c);
            pool_to_lds<NT, D>([&](int tt, float *x) { unpack_bf8(kw[tt], x); }, kbar, a, g, c);
        } else {
            pool_to_lds<NT, D>([&](int tt, float *x) { for (int s = 0; s < 8; ++s) x[s] = qr[tt][s]; },
                               qbar, a, g, c);
            pool_to_lds<NT, D>([&](int tt, float *x) { for (int s = 0; s < 8; ++s) x[s] = kr[tt][s]; },
                               kbar, a, g, c);
        }
        wave_sync();
        const f4 *kp = reinterpret_cast<const f4 *>(kbar + c * kLdStride + 8 * g);
        const f4 *qp = reinterpret_cast<const f4 *>(qbar + c * kLdStride + 8 * g);
        const f4 k0 = kp[0], k1 = kp[1], q0 = qp[0], q1 = qp[1];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            kb[s] = k0[s];
            kb[4 + s] = k1[s];
            qb[s] = q0[s];
            qb[4 + s] = q1[s];
        }
    }
    bf8 kbh, kbl, qbh, qbl;   // bf16 path: landmark rows as hi + lo terms
    if constexpr (BFM) {
        split_bf16(kb, kbh, kbl);
        split_bf16(qb, qbh, qbl);
    }
    const float s2u = a.s2 * a.inv_patch;    // one pooled side (S_L, S_U)
    const float s2a = s2u * a.inv_patch;     // both sides pooled (S_A)

    // ---- Step 3, G_U side: S_U^T tiles, row max over all N tokens, G_U^n.
    // guT[tt] lane (g,c): G_U^n[landmark c][token 16tt+4g+i].
    f4 guT[NT];
    float mu = -INFINITY;
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
        f4 acc = {0.f, 0.f, 0.f, 0.f};
        if constexpr (BFM) {
            acc = mfma_bf16(kw[tt], qbh, acc);
            acc = mfma_bf16(kw[tt], qbl, acc);
        } else {
#pragma unroll
            for (int s = 0; s < 8; ++s)
                acc = mfma4(kr[tt][s], qb[s], acc);
        }
        guT[tt] = acc;
        mu = fmaxf(mu, fmaxf(fmaxf(acc[0], acc[1]), fmaxf(acc[2], acc[3])));
    }
    mu = s2u * max_groups(mu);     // m_U of landmark c (base-2 units)
    float tden = 0.f;               // row sum of G_U^n (without a ones column)
#pragma unroll
    for (int tt = 0; tt < NT; ++tt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float e = (c < m) ? fast_exp2(fmaf(s2u, guT[tt][i], -mu)) : 0.f;
            guT[tt][i] = e;
            tden += e;
        }
    if constexpr (!PAD)
        tden = sum_groups(tden);

    // ---- Step 6, first product: T = G_U^n [V | 1]  (16 landmarks x 16 NCT).
    // T[ct] lane (g,c): T[landmark 4g+i][column 16ct+c].
    f4 T[NCT];
    if constexpr (BFM) {
        // token tiles in pairs: lane group g supplies tokens 4g..4g+3 of both
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
            T[ct] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int tp = 0; tp < (NT + 1) / 2; ++tp) {
            const int t1 = 2 * tp + 1;
            float g8[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                g8[i] = guT[2 * tp][i];
                g8[4 + i] = t1 < NT ? guT[t1 % NT][i] : 0.f;
            }
            bf8 gh, gl;
            split_bf16(g8, gh, gl);
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                uint16_t v8[8];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    v8[i] = vh[2 * tp][ct][i];
                    v8[4 + i] = t1 < NT ? vh[t1 % NT][ct][i] : uint16_t(0);
                }
                const bf8 vv = pack_bf8(v8);
                T[ct] = mfma_bf16(gh, vv, T[ct]);
                T[ct] = mfma_bf16(gl, vv, T[ct]);
            }
        }
    } else {
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
            f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int tt = 0; tt < NT; ++tt)
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    acc = mfma4(guT[tt][s], vr[tt][ct][s], acc);
            T[ct] = acc;
        }
    }

    // ---- Step 3, G_L side: S_L^T tiles, row max over landmarks, G_L^n.
    // glT[tt] lane (g,c): G_L^n[token 16tt+c][landmark 4g+i].
    f4 glT[NT];
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
        f4 acc = {0.f, 0.f, 0.f, 0.f};
        if constexpr (BFM) {
            acc = mfma_bf16(kbh, qw[tt], acc);
            acc = mfma_bf16(kbl, qw[tt], acc);
        } else {
#pragma unroll
            for (int s = 0; s < 8; ++s)
                acc = mfma4(kb[s], qr[tt][s], acc);
        }
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (4 * g + i < m)
                mx = fmaxf(mx, acc[i]);
        mx = s2u * max_groups(mx);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            glT[tt][i] = (4 * g + i < m) ? fast_exp2(fmaf(s2u, acc[i], -mx)) : 0.f;
    }

    // ---- Step 2: G_A^n (rows scaled by m_U).  AT lane (g,c): A[c][4g+i].
    f4 AT;
    {
        f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < 8; ++s)
            acc = mfma4(kb[s], qb[s], acc);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            AT[i] = (c < m && 4 * g + i < m) ? fast_exp2(fmaf(s2a, acc[i], -mu)) : 0.f;
    }

    // ---- Step 4: Z_0 = A^T / (||A||_1 ||A||_inf), then the iteration
    //      X = A Z;  Z <- Z (13I - X (15I - X (7I - X))) / 4.
    const float rowsum = sum_groups(AT[0] + AT[1] + AT[2] + AT[3]);   // sum_j A[c][j]
    const float colsum = fmaxf(fmaxf(sum_row(AT[0]), sum_row(AT[1])),  // max_i sum_r A[r][4g+i]
                               fmaxf(sum_row(AT[2]), sum_row(AT[3])));
    const float norm_inf = max_groups(max_row(rowsum));
    const float norm_1 = max_groups(colsum);
    const float alpha = 1.0f / (norm_1 * norm_inf);
    const f4 A = transpose16(AT, scr, g, c);
    f4 Z = AT * alpha, ZT = A * alpha;
    f4 eye;   // identity of the m x m block, D-layout
#pragma unroll
    for (int i = 0; i < 4; ++i)
        eye[i] = (4 * g + i == c && c < m) ? 1.f : 0.f;
    // The factor 1/4 of the update rides on A: with X' = (A/4) Z = X/4,
    //   4 Y1 = 28I - 16X',  Y2 = 15I - X' (4 Y1),  Y3 / 4 = 13I/4 - X' Y2,
    // and Z <- Z (Y3 / 4).  Scaling by powers of two is exact, so every value
    // equals the one of the update as written.  The constants ride in the
    // products' accumulators: -Y2 = X' (4 Y1) - 15I, Y3 / 4 = 13I/4 + X' (-Y2).
    const f4 ATq = AT * 0.25f, e28 = eye * 28.f, en15 = eye * -15.f, e13q = eye * 3.25f;
    if constexpr (BFM) {
        // bf16 inputs: every product as (hi + lo) x (hi + lo) bf16 terms; the
        // left factors come in both k orders, X'^T and Z^T by moving the split
        // terms of X' and Z through LDS.
        const SplitPair Aq = both_orders(split_tile(ATq).hl);
        auto step = [&]() {
            const bf8 zs = split_tile(Z).hl;
            const SplitPair ZTs = transpose_split(zs, scr, g, c);
            const f4 Xq = mm16_hl(Aq, zs);
            const bf8 xs = split_tile(Xq).hl;
            const SplitPair XTq = transpose_split(xs, scr, g, c);
            // Y2 = 15I - X (7I - X) = 15I - 28X' + 16X'^2, with X'^2 from the
            // split terms already at hand (no split of 4 Y1).
            const f4 X2 = mm16_hl(XTq, xs);
            f4 Y;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                Y[i] = fmaf(X2[i], -16.f, fmaf(Xq[i], 28.f, en15[i]));   // -Y2
            Y = mm16_hl(XTq, split_tile(Y).hl, e13q);   // 13I/4 - X' Y2
            Z = mm16_hl(ZTs, split_tile(Y).hl);
        };
        if constexpr (KF > 0) {
#pragma unroll
            for (int it = 0; it < KF; ++it)
                step();
        } else {
            for (int it = 0; it < a.iters; ++it)
                step();
        }
        if (KF > 0 || a.iters > 0)
            ZT = transpose16(Z, scr, g, c);
    } else {
        auto step = [&]() {
            const f4 Xq = mm16(ATq, Z);
            const f4 XTq = transpose16(Xq, scr, g, c);
            f4 Y;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                Y[i] = fmaf(Xq[i], -16.f, e28[i]);
            Y = mm16_acc(XTq, Y, en15);   // X' (4 Y1) - 15I = -Y2
            Y = mm16_acc(XTq, Y, e13q);   // 13I/4 - X' Y2
            Z = mm16(ZT, Y);
            ZT = transpose16(Z, scr, g, c);
        };
        if constexpr (KF > 0) {
#pragma unroll
            for (int it = 0; it < KF; ++it)
                step();
        } else {
            for (int it = 0; it < a.iters; ++it)
                step();
        }
    }

    // ---- Steps 5-6 re-associated: W = Z T (with the denominator column).
    f4 Wt[NCT];
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
        Wt[ct] = mm16(ZT, T[ct]);
    f4 wd = {0.f, 0.f, 0.f, 0.f};   // W_D[4g+i] (without a ones column)
    if constexpr (!PAD) {
        const f4 td = by_rows(tden, vec, g, c);                    // T_D[4g+i]
        const float wden =
            sum_groups(ZT[0] * td[0] + ZT[1] * td[1] + ZT[2] * td[2] + ZT[3] * td[3]);
        wd = by_rows(wden, vec, g, c);
    }
    // bf16 path: W as hi + lo terms, in both k orders.
    SplitPair ws[NCT];
    if constexpr (BFM) {
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
            ws[ct] = both_orders(split_tile(Wt[ct]).hl);
    }

    // ---- Steps 3 (G_L side), 6 and 7 per token tile: O = G_L^n W / O_D.
    const int olane = 4 * g * D + c;
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
        f4 on[NCT];
        bf8 gs;
        if constexpr (BFM)
            gs = split_tile(glT[tt]).hl;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
            if constexpr (BFM)
                on[ct] = mm16_lh(gs, ws[ct]);   // (G_hi + G_lo)(W_hi + W_lo)
            else
                on[ct] = mm16(glT[tt], Wt[ct]);
        }
        f4 rcp;   // 1 / O_D[16tt+4g+i]
        if constexpr (PAD) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                rcp[i] = __builtin_amdgcn_rcpf(row_bcast<D % 16>(on[NCT - 1][i]));
        } else {
            const float od = sum_groups(glT[tt][0] * wd[0] + glT[tt][1] * wd[1] +
                                        glT[tt][2] * wd[2] + glT[tt][3] * wd[3]);
            const f4 odr = by_rows(od, vec, g, c);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                rcp[i] = __builtin_amdgcn_rcpf(odr[i]);
        }
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
            f4 x;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                x[i] = on[ct][i] * rcp[i];
            // O straight to HBM, row-major.
            if constexpr (BFM) {
                // Rows (0, 1) and (2, 3) of this lane's feature are converted
                // in pairs (round to nearest even) and stored as 16-bit values.
                const int f = 16 * ct + c;
                if (f < D) {
                    const uint32_t p01 = pack_bf16x2(x[0], x[1]), p23 = pack_bf16x2(x[2], x[3]);
                    uint16_t *dst = reinterpret_cast<uint16_t *>(ou) + (16 * tt + 4 * g) * D + f;
                    dst[0] = uint16_t(p01);
                    dst[D] = uint16_t(p01 >> 16);
                    dst[2 * D] = uint16_t(p23);
                    dst[3 * D] = uint16_t(p23 >> 16);
                }
            } else {
                if (16 * ct + c < D) {
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        ou[olane + (16 * tt + i) * D + 16 * ct] = x[i];
                }
            }
        }
    }
}

// ---- 64-token windows, few units: one unit per four-wave workgroup --------
//
// When the units are fewer than the SIMDs, one wave per unit leaves most of
// the chip idle and the launch lasts one unit's whole dependent chain.  Here
// the four waves of a workgroup split the unit's four token tiles: wave w
// loads tile w of Q, K and V, and the passes over tokens are shared through
// LDS -- the staged rows for Step 1, the per-wave maxima of S_U and the
// per-wave partial sums T_w = G_U^n [V | 1] over the wave's keys (Step 3, G_U
// side; only the order of the additions changes).  Wave 0 then runs Step 2,
// the pseudo-inverse and W = Z T (the other waves wait), and every wave forms
// Steps 3 (G_L side), 6 and 7 for its own tile.  Fixed 8 x 8 pooling grids
// only (their patches never straddle a token tile).

template <class E, int D>
struct MwLds {
    static constexpr int NCT = (D + 15) / 16;
    static constexpr int RS = raw_stride<E>();
    static constexpr int qst = 0;                          // [64][RS] raw Q chunks
    static constexpr int kst = qst + 64 * RS;              // [64][RS] raw K chunks
    static constexpr int xm = kst + 64 * RS;               // [4][16] maxima of S_U per wave
    static constexpr int xd = xm + 64;                     // [4][16] T_D per wave
    static constexpr int xt = xd + 64;                     // [4][NCT][64 lanes][4] T per wave
    static constexpr int wt = xt + 4 * NCT * 256;          // [NCT][64][4] W, then [64][4] W_D
    static constexpr int scr = wt + NCT * 256 + 256;       // wave 0's transpose scratch
    static constexpr int vec = scr + 16 * kTrStride;       // [4][64] row vectors
    static constexpr int total = vec + 4 * 64;
};

template <class E, int D, bool BFM, int GRID, int KF>
__global__ void __launch_bounds__(256)
tiled_small_mw_kernel(const typename E::T *__restrict__ q, const typename E::T *__restrict__ k,
                      const typename E::T *__restrict__ v, typename E::T *__restrict__ o,
                      SmallArgs a)
{
    static_assert(GRID != kGridAny, "the fixed 8 x 8 grids keep a patch inside a token tile");
    constexpr int N = 64;
    using L = MwLds<E, D>;
    constexpr int NCT = L::NCT;
    constexpr bool PAD = D % 16 != 0;
    extern __shared__ __attribute__((aligned(16))) float lds[];
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int g = lane >> 4, c = lane & 15;
    const int m = GRID == kGrid2x2 ? 16 : 8;
    float *vec = lds + L::vec + 64 * w;
    const int64_t base = int64_t(blockIdx.x) * N * D;
    const typename E::T *qu = q + base, *ku = k + base, *vu = v + base;
    typename E::T *ou = o + base;

    // ---- loads of this wave's token tile w
    const int off = (16 * w + c) * D + chunk_start<D>(g);
    float qr[8], kr[8];
    bf8 qw, kw;
    if constexpr (BFM) {
        qw = load_row8_bf16(reinterpret_cast<const uint16_t *>(qu) + off);
        kw = load_row8_bf16(reinterpret_cast<const uint16_t *>(ku) + off);
    } else {
        load_row8<D>(qu + off, qr);
        load_row8<D>(ku + off, kr);
    }
    // V rows 16w+4g+s of column 16ct+c (the ones column at column D)
    float vr[NCT][4];
    uint16_t vh[NCT][4];
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) {
        const int f = 16 * ct + c;
        const int vlane = (16 * w + 4 * g) * D + min(f, D - 1);
        const bool ones = PAD && ct == NCT - 1 && f == D;
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            if constexpr (BFM) {
                const uint16_t y = reinterpret_cast<const uint16_t *>(vu)[vlane + x * D];
                vh[ct][x] = ones ? uint16_t(0x3F80) : y;
            } else {
                const float y = E::load(vu, vlane + x * D);
                vr[ct][x] = ones ? 1.f : y;
            }
        }
    }

    // ---- Step 1: every wave stages its rows; every wave forms the patch sums.
    float qb[8], kb[8];
    if constexpr (BFM) {
        stage_chunk<E>(qw, lds + L::qst, w, g, c);
        stage_chunk<E>(kw, lds + L::kst, w, g, c);
    } else {
        stage_chunk<E>(qr, lds + L::qst, w, g, c);
        stage_chunk<E>(kr, lds + L::kst, w, g, c);
    }
    __syncthreads();
    patch_sums<E, D, GRID>(lds + L::qst, qb, m, g, c);
    patch_sums<E, D, GRID>(lds + L::kst, kb, m, g, c);
    bf8 kbh, kbl, qbh, qbl;
    if constexpr (BFM) {
        split_bf16(kb, kbh, kbl);
        split_bf16(qb, qbh, qbl);
    }
    const float s2u = a.s2 * a.inv_patch;    // one pooled side (S_L, S_U)
    const float s2a = s2u * a.inv_patch;     // both sides pooled (S_A)

    // ---- Step 3, G_U side over this wave's keys; the row maxima over all
    // keys come from the four waves' maxima.
    f4 su = {0.f, 0.f, 0.f, 0.f};   // lane (g,c): S_U[landmark c][key 16w+4g+i]
    if constexpr (BFM) {
        su = mfma_bf16(kw, qbh, su);
        su = mfma_bf16(kw, qbl, su);
    } else {
#pragma unroll
        for (int x = 0; x < 8; ++x)
            su = mfma4(kr[x], qb[x], su);
    }
    {
        const float mw = max_groups(fmaxf(fmaxf(su[0], su[1]), fmaxf(su[2], su[3])));
        if (g == 0)
            lds[L::xm + 16 * w + c] = mw;
    }
    // ---- Step 3, G_L side for this wave's query tile (no exchange needed).
    // glT lane (g,c): G_L^n[token 16w+c][landmark 4g+i].
    f4 glT;
    {
        f4 acc = {0.f, 0.f, 0.f, 0.f};
        if constexpr (BFM) {
            acc = mfma_bf16(kbh, qw, acc);
            acc = mfma_bf16(kbl, qw, acc);
        } else {
#pragma unroll
            for (int x = 0; x < 8; ++x)
                acc = mfma4(kb[x], qr[x], acc);
        }
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (4 * g + i < m)
                mx = fmaxf(mx, acc[i]);
        mx = s2u * max_groups(mx);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            glT[i] = (4 * g + i < m) ? fast_exp2(fmaf(s2u, acc[i], -mx)) : 0.f;
    }
    __syncthreads();   // the waves' maxima
    float mu = lds[L::xm + c];
#pragma unroll
    for (int u = 1; u < 4; ++u)
        mu = fmaxf(mu, lds[L::xm + 16 * u + c]);
    mu *= s2u;   // m_U of landmark c (base-2 units)
    float tden = 0.f;
    f4 e;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        e[i] = (c < m) ? fast_exp2(fmaf(s2u, su[i], -mu)) : 0.f;
        tden += e[i];
    }
    // T_w = G_U^n [V | 1] over this wave's 16 keys: T[ct] lane (g,c) holds
    // T_w[landmark 4g+i][column 16ct+c].
    f4 T[NCT];
    if constexpr (BFM) {
        // the bf16 product contracts 32 keys: this tile's, then 16 zeros
        float g8[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            g8[i] = e[i];
            g8[4 + i] = 0.f;
        }
        bf8 gh, gl;
        split_bf16(g8, gh, gl);
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
            const uint16_t v8[8] = {vh[ct][0], vh[ct][1], vh[ct][2], vh[ct][3], 0, 0, 0, 0};
            const bf8 vv = pack_bf8(v8);
            T[ct] = mfma_bf16(gh, vv, f4{0.f, 0.f, 0.f, 0.f});
            T[ct] = mfma_bf16(gl, vv, T[ct]);
        }
    } else {
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
            f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int x = 0; x < 4; ++x)
                acc = mfma4(e[x], vr[ct][x], acc);
            T[ct] = acc;
        }
    }
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
        reinterpret_cast<f4 *>(lds + L::xt + (w * NCT + ct) * 256)[lane] = T[ct];
    if constexpr (!PAD) {
        tden = sum_groups(tden);
        if (g == 0)
            lds[L::xd + 16 * w + c] = tden;
    }
    __syncthreads();   // the waves' partial sums

    if (w == 0) {
        // T and T_D of the unit: the four waves' sums, in wave order.
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
            f4 acc = reinterpret_cast<const f4 *>(lds + L::xt + ct * 256)[lane];
#pragma unroll
            for (int u = 1; u < 4; ++u)
                acc += reinterpret_cast<const f4 *>(lds + L::xt + (u * NCT + ct) * 256)[lane];
            T[ct] = acc;
        }
        if constexpr (!PAD)
            tden = lds[L::xd + c] + lds[L::xd + 16 + c] + lds[L::xd + 32 + c] +
                   lds[L::xd + 48 + c];
        float *scr = lds + L::scr;
        // ---- Step 2: G_A^n.  AT lane (g,c): A[c][4g+i].
        f4 AT;
        {
            f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int x = 0; x < 8; ++x)
                acc = mfma4(kb[x], qb[x], acc);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                AT[i] = (c < m && 4 * g + i < m) ? fast_exp2(fmaf(s2a, acc[i], -mu)) : 0.f;
        }
        // ---- Step 4, as in the one-wave kernel.
        const float rowsum = sum_groups(AT[0] + AT[1] + AT[2] + AT[3]);
        const float colsum = fmaxf(fmaxf(sum_row(AT[0]), sum_row(AT[1])),
                                   fmaxf(sum_row(AT[2]), sum_row(AT[3])));
        const float norm_inf = max_groups(max_row(rowsum));
        const float norm_1 = max_groups(colsum);
        const float alpha = 1.0f / (norm_1 * norm_inf);
        const f4 A = transpose16(AT, scr, g, c);
        f4 Z = AT * alpha, ZT = A * alpha;
        f4 eye;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            eye[i] = (4 * g + i == c && c < m) ? 1.f : 0.f;
        const f4 ATq = AT * 0.25f, e28 = eye * 28.f, en15 = eye * -15.f, e13q = eye * 3.25f;
        if constexpr (BFM) {
            const SplitPair Aq = both_orders(split_tile(ATq).hl);
            auto step = [&]() {
                const bf8 zs = split_tile(Z).hl;
                const SplitPair ZTs = transpose_split(zs, scr, g, c);
                const f4 Xq = mm16_hl(Aq, zs);
                const bf8 xs = split_tile(Xq).hl;
                const SplitPair XTq = transpose_split(xs, scr, g, c);
                const f4 X2 = mm16_hl(XTq, xs);
                f4 Y;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    Y[i] = fmaf(X2[i], -16.f, fmaf(Xq[i], 28.f, en15[i]));   // -Y2
                Y = mm16_hl(XTq, split_tile(Y).hl, e13q);   // 13I/4 - X' Y2
                Z = mm16_hl(ZTs, split_tile(Y).hl);
            };
            if constexpr (KF > 0) {
#pragma unroll
                for (int it = 0; it < KF; ++it)
                    step();
            } else {
                for (int it = 0; it < a.iters; ++it)
                    step();
            }
            if (KF > 0 || a.iters > 0)
                ZT = transpose16(Z, scr, g, c);
        } else {
            auto step = [&]() {
                const f4 Xq = mm16(ATq, Z);
                const f4 XTq = transpose16(Xq, scr, g, c);
                f4 Y;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    Y[i] = fmaf(Xq[i], -16.f, e28[i]);
                Y = mm16_acc(XTq, Y, en15);   // X' (4 Y1) - 15I = -Y2
                Y = mm16_acc(XTq, Y, e13q);   // 13I/4 - X' Y2
                Z = mm16(ZT, Y);
                ZT = transpose16(Z, scr, g, c);
            };
            if constexpr (KF > 0) {
#pragma unroll
                for (int it = 0; it < KF; ++it)
                    step();
            } else {
                for (int it = 0; it < a.iters; ++it)
                    step();
            }
        }
        // ---- Steps 5-6 re-associated: W = Z T, published for every wave.
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
            reinterpret_cast<f4 *>(lds + L::wt + ct * 256)[lane] = mm16(ZT, T[ct]);
        if constexpr (!PAD) {
            const f4 td = by_rows(tden, vec, g, c);
            const float wden =
                sum_groups(ZT[0] * td[0] + ZT[1] * td[1] + ZT[2] * td[2] + ZT[3] * td[3]);
            reinterpret_cast<f4 *>(lds + L::wt + NCT * 256)[lane] = by_rows(wden, vec, g, c);
        }
    }
    __syncthreads();   // W

    // ---- Steps 3 (G_L side), 6 and 7 for this wave's tile.
    f4 Wt[NCT];
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
        Wt[ct] = reinterpret_cast<const f4 *>(lds + L::wt + ct * 256)[lane];
    f4 on[NCT];
    if constexpr (BFM) {
        const bf8 gs = split_tile(glT).hl;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
            on[ct] = mm16_lh(gs, both_orders(split_tile(Wt[ct]).hl));
    } else {
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
            on[ct] = mm16(glT, Wt[ct]);
    }
    f4 rcp;   // 1 / O_D[16w+4g+i]
    if constexpr (PAD) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            rcp[i] = __builtin_amdgcn_rcpf(row_bcast<D % 16>(on[NCT - 1][i]));
    } else {
        const f4 wd = reinterpret_cast<const f4 *>(lds + L::wt + NCT * 256)[lane];
        const float od = sum_groups(glT[0] * wd[0] + glT[1] * wd[1] + glT[2] * wd[2] +
                                    glT[3] * wd[3]);
        const f4 odr = by_rows(od, vec, g, c);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            rcp[i] = __builtin_amdgcn_rcpf(odr[i]);
    }
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) {
        const int f = 16 * ct + c;
        if (f < D) {
            f4 x;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                x[i] = on[ct][i] * rcp[i];
            if constexpr (BFM) {
                const uint32_t p01 = pack_bf16x2(x[0], x[1]), p23 = pack_bf16x2(x[2], x[3]);
                uint16_t *dst = reinterpret_cast<uint16_t *>(ou) + (16 * w + 4 * g) * D + f;
                dst[0] = uint16_t(p01);
                dst[D] = uint16_t(p01 >> 16);
                dst[2 * D] = uint16_t(p23);
                dst[3 * D] = uint16_t(p23 >> 16);
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    ou[(16 * w + 4 * g + i) * D + f] = x[i];
            }
        }
    }
}

bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

int ilog2(int x)
{
    int r = 0;
    while ((1 << r) < x)
        ++r;
    return r;
}

// Below this many units, four-wave workgroups would leave compute units idle
// (256 on the MI355X): each unit then gets a workgroup of its own, so that the
// units spread over the whole chip.
constexpr int64_t kFewUnits = 4 * 256;

template <class E, int NT, int D, int GRID = kGridAny, int KF = 0>
void launch_small(const Problem &p, const SmallArgs &a, hipStream_t stream)
{
    if constexpr (NT == 4 && GRID != kGridAny) {
        if (p.units < kFewUnits) {   // one unit per four-wave workgroup
            const size_t lds = size_t(MwLds<E, D>::total) * sizeof(float);
            hipLaunchKernelGGL((tiled_small_mw_kernel<E, D, E::bytes == 2, GRID, KF>),
                               dim3(unsigned(p.units)), dim3(256), lds, stream,
                               static_cast<const typename E::T *>(p.q),
                               static_cast<const typename E::T *>(p.k),
                               static_cast<const typename E::T *>(p.v),
                               static_cast<typename E::T *>(p.o), a);
            return;
        }
    }
    const int wpb = p.units < kFewUnits ? 1 : kWavesPerBlock;
    const unsigned blocks = unsigned((p.units + wpb - 1) / wpb);
    const size_t lds = size_t(wpb) * SmallLds<E, NT, D, GRID>::kPerWave * sizeof(float);
    hipLaunchKernelGGL((tiled_small_kernel<E, NT, D, E::bytes == 2, GRID, KF>), dim3(blocks),
                       dim3(64 * wpb), lds, stream, static_cast<const typename E::T *>(p.q),
                       static_cast<const typename E::T *>(p.k),
                       static_cast<const typename E::T *>(p.v),
                       static_cast<typename E::T *>(p.o), a);
}

template <class E, int D>
void launch_small_d(const Problem &p, const SmallArgs &a, hipStream_t stream)
{
    switch (p.N) {
    case 16: launch_small<E, 1, D>(p, a, stream); break;
    case 32: launch_small<E, 2, D>(p, a, stream); break;
    default:
        switch (grid_of(a, p.N)) {
        // K = 6, the iteration count of the paper's experiments, unrolled.
        case kGrid2x2:
            if (a.iters == 6)
                launch_small<E, 4, D, kGrid2x2, 6>(p, a, stream);
            else
                launch_small<E, 4, D, kGrid2x2>(p, a, stream);
            break;
        case kGrid2x4:
            if (a.iters == 6)
                launch_small<E, 4, D, kGrid2x4, 6>(p, a, stream);
            else
                launch_small<E, 4, D, kGrid2x4>(p, a, stream);
            break;
        default: launch_small<E, 4, D>(p, a, stream); break;
        }
        break;
    }
}

template <class E>
void launch_small_e(const Problem &p, const SmallArgs &a, hipStream_t stream)
{
    switch (p.d) {
    case 8: launch_small_d<E, 8>(p, a, stream); break;
    case 12: launch_small_d<E, 12>(p, a, stream); break;
    case 16: launch_small_d<E, 16>(p, a, stream); break;
    case 20: launch_small_d<E, 20>(p, a, stream); break;
    case 24: launch_small_d<E, 24>(p, a, stream); break;
    case 28: launch_small_d<E, 28>(p, a, stream); break;
    case 30: launch_small_d<E, 30>(p, a, stream); break;
    default: launch_small_d<E, 32>(p, a, stream); break;
    }
}

bool small_supported(const Problem &p)
{
    const Geometry &g = p.geo;
    if (!(p.N == 16 || p.N == 32 || p.N == 64) || p.m > 16 || !tiled_width(p.d))
        return false;
    if (!is_pow2(g.cols) || !is_pow2(g.pr) || !is_pow2(g.pc) || !is_pow2(g.gc))
        return false;
    // bf16 row chunks of Q and K are read as 16-byte pieces that start at even
    // elements, and O is written in pairs of features.
    if (p.dtype == 1 && (uintptr_t(p.q) | uintptr_t(p.k) | uintptr_t(p.o)) % 4 != 0)
        return false;
    return true;
}

}  // namespace

bool tiled_supported(const Problem &p) { return small_supported(p) || tiled_large_supported(p); }

hipError_t launch_tiled_forward(const Problem &p, hipStream_t stream)
{
    if (!small_supported(p))
        return launch_tiled_large(p, stream);
    SmallArgs a;
    a.units = p.units;
    a.m = p.m;
    a.iters = p.iters;
    a.s2 = p.scale * kLog2e;
    a.inv_patch = 1.0f / float(p.geo.pr * p.geo.pc);
    a.lg_cols = ilog2(p.geo.cols);
    a.lg_pr = ilog2(p.geo.pr);
    a.lg_pc = ilog2(p.geo.pc);
    a.lg_gc = ilog2(p.geo.gc);
    a.free_bits = (p.geo.pc - 1) | ((p.geo.pr - 1) * p.geo.cols);
    if (p.dtype == 0)
        launch_small_e<F32>(p, a, stream);
    else
        launch_small_e<BF16>(p, a, stream);
    return hipGetLastError();
}

}  // namespace nystra
