// Helpers shared by the MFMA-tiled kernels: the 16x16 register tile
// convention, cross-lane exchanges and branch-free feature-chunk loads.
//
// Register tile convention ("D-layout").  A 16x16 fp32 tile M lives in one
// float4 per lane: lane (g = lane / 16, c = lane % 16) holds M[4g + i][c],
// i = 0..3 -- the layout in which v_mfma_f32_16x16x4f32 returns its result.
// Running a 16-deep contraction as four MFMA steps in which lane group g
// supplies the k-index 4g + s at step s, a D-layout tile can be fed back
// directly:  mm16(LT, R) = L * R  when LT holds L^T and R holds R, both in
// D-layout.  A product's result is immediately the right-hand operand of the
// next product, and a matrix is usable as a left-hand operand once its
// transpose is in D-layout.
#pragma once

#include "device_common.hpp"

namespace nystra {
namespace tile {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kLdStride = 36;   // row stride (floats) of the landmark tiles in LDS
constexpr int kTrStride = 20;   // row stride (floats) of the transpose scratch

__device__ inline f4 mfma4(float a, float b, f4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// L * R for 16x16 tiles, LT = L^T and R in D-layout.
__device__ inline f4 mm16(f4 LT, f4 R)
{
    f4 acc = {0.f, 0.f, 0.f, 0.f};
    acc = mfma4(LT[0], R[0], acc);
    acc = mfma4(LT[1], R[1], acc);
    acc = mfma4(LT[2], R[2], acc);
    acc = mfma4(LT[3], R[3], acc);
    return acc;
}

// acc + L * R, chaining the accumulator through the matrix core.
__device__ inline f4 mm16_acc(f4 LT, f4 R, f4 acc)
{
    acc = mfma4(LT[0], R[0], acc);
    acc = mfma4(LT[1], R[1], acc);
    acc = mfma4(LT[2], R[2], acc);
    acc = mfma4(LT[3], R[3], acc);
    return acc;
}

// ---- bf16 matrix-core operands --------------------------------------------
// v_mfma_f32_16x16x32_bf16: lane (g, c) supplies A[c][8g + j] and B[8g + j][c]
// (j = 0..7) and receives D[4g + i][c].  An fp32 operand x is carried as two
// bf16 terms, hi = bf16(x) and lo = bf16(x - hi), which keep ~16 bits.

typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

__device__ inline f4 mfma_bf16(bf8 a, bf8 b, f4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

struct __attribute__((aligned(4))) U16B {
    uint32_t w[4];
};

// A D-layout fp32 tile as two bf16 terms, packed as the A operand of a
// 16x16x32 product over a 16-deep contraction: lane group g supplies, at
// k = 8g + j, the hi term (j < 4) or the lo term (j >= 4) of its element
// 4g + (j & 3).  hi = bf16(x) and lo = bf16(x - hi) (round to nearest even).
struct SplitTile {
    bf8 hl;   // [hi0..hi3, lo0..lo3]
};

__device__ inline uint32_t cvt_bf16x2(float lo, float hi)
{
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2{lo, hi}), b2));   // RNE
}

// The residuals x - hi of a converted pair, one v_dot2_f32_bf16 each:
// x0 + (-1) hi0 + 0 hi1 and x1 + 0 hi0 + (-1) hi1.  Every partial result is
// exact (hi is x rounded to 8 bits, so x - hi is an fp32 value), so these are
// the values of the subtractions x - float(hi), without widening hi first.
// The selectors (-1, 0) and (0, -1) come from SALU moves the compiler cannot
// fold: as a literal, 0xbf800000 would be encoded as the fp32 inline
// constant -1.0, which a packed bf16 operand does not read as (0, -1).
struct NegSel {
    uint32_t s0, s1;
};

__device__ inline NegSel neg_selectors()
{
    uint32_t a, b;
    asm("s_mov_b32 %0, 0xbf80" : "=s"(a));
    asm("s_mov_b32 %0, 0xbf800000" : "=s"(b));
    return NegSel{a, b};
}

__device__ inline uint32_t residual_bf16x2(uint32_t h, float x0, float x1, NegSel s)
{
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    const b2 hv = __builtin_bit_cast(b2, h);
    const float l0 = __builtin_amdgcn_fdot2_f32_bf16(hv, __builtin_bit_cast(b2, s.s0), x0, false);
    const float l1 = __builtin_amdgcn_fdot2_f32_bf16(hv, __builtin_bit_cast(b2, s.s1), x1, false);
    return cvt_bf16x2(l0, l1);
}

// Eight fp32 values as hi = bf16(x) and lo = bf16(x - hi), both rounded to
// nearest even, converted in pairs.
__device__ inline void split_bf16(const float (&x)[8], bf8 &hi, bf8 &lo)
{
    const NegSel s = neg_selectors();
    U16B h, l;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        h.w[p] = cvt_bf16x2(x[2 * p], x[2 * p + 1]);
        l.w[p] = residual_bf16x2(h.w[p], x[2 * p], x[2 * p + 1], s);
    }
    hi = __builtin_bit_cast(bf8, h);
    lo = __builtin_bit_cast(bf8, l);
}

__device__ inline SplitTile split_tile(f4 x)
{
    const NegSel s = neg_selectors();
    U16B u;
    u.w[0] = cvt_bf16x2(x[0], x[1]);
    u.w[1] = cvt_bf16x2(x[2], x[3]);
    u.w[2] = residual_bf16x2(u.w[0], x[0], x[1], s);
    u.w[3] = residual_bf16x2(u.w[1], x[2], x[3], s);
    return SplitTile{__builtin_bit_cast(bf8, u)};
}

// A split tile in both orders of its k slots: hl = [hi | lo] (the packing of
// SplitTile) and lh = [lo | hi].
struct SplitPair {
    bf8 hl, lh;
};

__device__ inline SplitPair both_orders(bf8 hl)
{
    const U16B u = __builtin_bit_cast(U16B, hl);
    const U16B v = {{u.w[2], u.w[3], u.w[0], u.w[1]}};
    return SplitPair{hl, __builtin_bit_cast(bf8, v)};
}

// L * R for 16x16 tiles with both factors split into bf16 hi + lo terms, on
// the bf16 matrix cores with fp32 accumulation.  Pairing [hi | lo] with
// [hi | lo] gives L_hi R_hi + L_lo R_lo; pairing [lo | hi] with [hi | lo]
// gives the two cross terms; together the full product of the two sums.
// mm16_hl takes LT = L^T in both orders (and adds acc), mm16_lh R in both orders.
__device__ inline f4 mm16_hl(const SplitPair &LT, bf8 R, f4 acc = f4{0.f, 0.f, 0.f, 0.f})
{
    acc = mfma_bf16(LT.hl, R, acc);
    return mfma_bf16(LT.lh, R, acc);
}

__device__ inline f4 mm16_lh(bf8 LT, const SplitPair &R)
{
    const f4 acc = mfma_bf16(LT, R.hl, f4{0.f, 0.f, 0.f, 0.f});
    return mfma_bf16(LT, R.lh, acc);
}

// Orders the LDS traffic of one wavefront (all lanes execute in lockstep, so
// only the compiler and the memory counters need fencing).
__device__ inline void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// D-layout transpose through the wave's LDS scratch.
__device__ inline f4 transpose16(f4 M, float *scr, int g, int c)
{
#pragma unroll
    for (int i = 0; i < 4; ++i)
        scr[(4 * g + i) * kTrStride + c] = M[i];
    wave_sync();
    f4 r = *reinterpret_cast<const f4 *>(scr + c * kTrStride + 4 * g);
    wave_sync();
    return r;
}

// Transpose of a split D-layout tile through the wave's LDS scratch (at least
// 16 * kTrStride floats): the bf16 terms move as 16-bit values, so the split
// of M^T costs no arithmetic.  Element (r, col) of plane p (0 = hi, 1 = lo)
// sits at bf16 index r * 40 + (col / 4) * 8 + 4p + col % 4, so that a lane
// reads its [hi | lo] chunk of a transposed row with one 16-byte load.
__device__ inline SplitPair transpose_split(bf8 s, float *scr, int g, int c)
{
    static_assert(16 * 40 * 2 <= 16 * kTrStride * 4, "scratch holds both planes");
    uint16_t *b = reinterpret_cast<uint16_t *>(scr);
    const U16B u = __builtin_bit_cast(U16B, s);
    const int col = (c >> 2) * 8 + (c & 3);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int at = (4 * g + i) * 40 + col;
        b[at] = uint16_t(u.w[i >> 1] >> (16 * (i & 1)));
        b[at + 4] = uint16_t(u.w[2 + (i >> 1)] >> (16 * (i & 1)));
    }
    wave_sync();
    const uint16_t *row = b + c * 40 + 8 * g;
    const U16B hl = *reinterpret_cast<const U16B *>(row);
    typedef uint32_t u2 __attribute__((ext_vector_type(2)));
    const u2 h = *reinterpret_cast<const u2 *>(row), l = *reinterpret_cast<const u2 *>(row + 4);
    wave_sync();
    const U16B lh = {{l[0], l[1], h[0], h[1]}};
    return SplitPair{__builtin_bit_cast(bf8, hl), __builtin_bit_cast(bf8, lh)};
}

// Per-token vector exchange: value x (held per lane column c, identical in
// all four lane groups) returned at row positions 4g + i.
__device__ inline f4 by_rows(float x, float *vec, int g, int c)
{
    if (g == 0)
        vec[c] = x;
    wave_sync();
    f4 r = *reinterpret_cast<const f4 *>(vec + 4 * g);
    wave_sync();
    return r;
}

// ---- cross-lane operations (wave64; a "row" is 16 lanes) ------------------
// DPP forms fuse into the consuming VALU instruction and the permlane swaps
// are VALU instructions; the swizzle goes through the LDS crossbar without
// touching LDS memory.

__device__ inline float dpp_xor1(float x) { return __builtin_amdgcn_update_dpp(0.f, x, 0xB1, 0xF, 0xF, false); }
__device__ inline float dpp_xor2(float x) { return __builtin_amdgcn_update_dpp(0.f, x, 0x4E, 0xF, 0xF, false); }
// Row rotations read a valid lane everywhere, so bound_ctrl is immaterial;
// setting it lets the compiler fold the move into the consuming instruction.
__device__ inline float dpp_ror4(float x) { return __builtin_amdgcn_update_dpp(0.f, x, 0x124, 0xF, 0xF, true); }
// Rotating a 16-lane row by 8 is the exchange of lanes c and c ^ 8.
__device__ inline float dpp_xor8(float x) { return __builtin_amdgcn_update_dpp(0.f, x, 0x128, 0xF, 0xF, true); }

// Every lane of a 16-lane row receives the value of that row's lane SRC
// (DPP row_newbcast, a VALU operand modifier).
template <int SRC>
__device__ inline float row_bcast(float x)
{
    static_assert(SRC >= 0 && SRC < 16, "source lane within the row");
    return __builtin_amdgcn_update_dpp(0.f, x, 0x150 + SRC, 0xF, 0xF, true);
}
__device__ inline float swz_xor4(float x)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x101F));
}

// Pairs (x[l], x[l ^ 16]) and (x[l], x[l ^ 32]) in VALU registers: the
// permlane swaps of a value with itself leave, in every lane, the row (half)
// of the pair with the lower index in .first and the other in .second.
struct LanePair {
    float first, second;
};

__device__ inline LanePair pair_xor16(float x)
{
    const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(unsigned, x),
                                                    __builtin_bit_cast(unsigned, x), false, false);
    return LanePair{__builtin_bit_cast(float, unsigned(r[0])), __builtin_bit_cast(float, unsigned(r[1]))};
}

__device__ inline LanePair pair_xor32(float x)
{
    const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, x),
                                                    __builtin_bit_cast(unsigned, x), false, false);
    return LanePair{__builtin_bit_cast(float, unsigned(r[0])), __builtin_bit_cast(float, unsigned(r[1]))};
}

// Sum / max over the four lanes c, c^16, c^32, c^48 (the lane groups g);
// every lane gets the same bits.
__device__ inline float sum_groups(float x)
{
    const LanePair a = pair_xor16(x);
    const LanePair b = pair_xor32(a.first + a.second);
    return b.first + b.second;
}

__device__ inline float max_groups(float x)
{
    const LanePair a = pair_xor16(x);
    const LanePair b = pair_xor32(fmaxf(a.first, a.second));
    return fmaxf(b.first, b.second);
}

// Sum / max over the 16 lanes of a row.
__device__ inline float sum_row(float x)
{
    x += dpp_xor1(x);
    x += dpp_xor2(x);
    x += dpp_ror4(x);
    return x + dpp_xor8(x);
}

__device__ inline float max_row(float x)
{
    x = fmaxf(x, dpp_xor1(x));
    x = fmaxf(x, dpp_xor2(x));
    x = fmaxf(x, dpp_ror4(x));
    return fmaxf(x, dpp_xor8(x));
}


// Feature chunk of lane group g.  The contraction over features runs as
// eight MFMA steps in which group g supplies the features in slots s = 0..7.
// Slot s of group g holds feature f0(g) + s with f0(g) = min(8g, D - 8), so a
// chunk never reaches past its row; slots whose feature belongs to a lower
// group (f0 + s < 8g) are zeroed.  D (>= 8) is a compile-time constant, so
// every load is in bounds and the masks are plain selects.
template <int D>
__device__ inline int chunk_start(int g) { return min(8 * g, D - 8); }

template <int D>
__device__ inline bool slot_valid(int g, int s) { return chunk_start<D>(g) + s >= 8 * g; }

template <class E, int D>
__device__ inline void load_chunk8(const typename E::T *row, int g, float *out)
{
    static_assert(D >= 8, "tiled kernel needs at least 8 features");
    const int f0 = chunk_start<D>(g);
    if constexpr (E::bytes == 4) {
        const U16B a = *reinterpret_cast<const U16B *>(row + f0);
        const U16B b = *reinterpret_cast<const U16B *>(row + f0 + 4);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            out[j] = slot_valid<D>(g, j) ? __uint_as_float(a.w[j]) : 0.f;
            out[4 + j] = slot_valid<D>(g, 4 + j) ? __uint_as_float(b.w[j]) : 0.f;
        }
    } else {
        const U16B a = *reinterpret_cast<const U16B *>(row + f0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            out[2 * j] = slot_valid<D>(g, 2 * j) ? __uint_as_float(a.w[j] << 16) : 0.f;
            out[2 * j + 1] =
                slot_valid<D>(g, 2 * j + 1) ? __uint_as_float(a.w[j] & 0xffff0000u) : 0.f;
        }
    }
}

// Eight features of one bf16 row as raw bits, in the slot layout of
// load_chunk8 (D is even, so invalid slots come in whole 32-bit pairs).
template <int D>
__device__ inline bf8 load_chunk8_bf8(const uint16_t *row, int g)
{
    U16B u = *reinterpret_cast<const U16B *>(row + chunk_start<D>(g));
#pragma unroll
    for (int j = 0; j < 4; ++j)
        if (!slot_valid<D>(g, 2 * j))
            u.w[j] = 0u;
    return __builtin_bit_cast(bf8, u);
}

// A raw bf16 chunk (load_row8_bf16 at chunk_start) with the slots that a
// lower lane group carries zeroed: the load_chunk8_bf8 result, applied after
// the load so that a prefetched chunk is not waited for at its issue.
template <int D>
__device__ inline bf8 mask_chunk8_bf8(bf8 x, int g)
{
    U16B u = __builtin_bit_cast(U16B, x);
#pragma unroll
    for (int j = 0; j < 4; ++j)
        if (!slot_valid<D>(g, 2 * j))
            u.w[j] = 0u;
    return __builtin_bit_cast(bf8, u);
}

// Slot s of lane group g carries a feature that no lower group carries; the
// chunk of the last, partial group (f0 = D - 8) overlaps the one below it.
// Equivalent to slot_valid, written so that D-dependent parts fold.
template <int D>
__device__ inline bool slot_keep(int g, int s)
{
    if constexpr (D % 8 == 0)
        return g < D / 8;
    else
        return s >= 8 - D % 8 ? g <= D / 8 : g < D / 8;
}

// The eight row elements of a chunk, unmasked (overlapping slots included).
template <int D>
__device__ inline void load_row8(const float *p, float *out)
{
    const U16B a = *reinterpret_cast<const U16B *>(p);
    const U16B b = *reinterpret_cast<const U16B *>(p + 4);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        out[j] = __uint_as_float(a.w[j]);
        out[4 + j] = __uint_as_float(b.w[j]);
    }
}

__device__ inline bf8 load_row8_bf16(const uint16_t *p)
{
    return __builtin_bit_cast(bf8, *reinterpret_cast<const U16B *>(p));
}

__device__ inline void unpack_bf8(bf8 v, float *out)
{
    const U16B u = __builtin_bit_cast(U16B, v);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        out[2 * j] = __uint_as_float(u.w[j] << 16);
        out[2 * j + 1] = __uint_as_float(u.w[j] & 0xffff0000u);
    }
}

__device__ inline bf8 pack_bf8(const uint16_t (&x)[8])
{
    U16B u;
#pragma unroll
    for (int j = 0; j < 4; ++j)
        u.w[j] = uint32_t(x[2 * j]) | (uint32_t(x[2 * j + 1]) << 16);
    return __builtin_bit_cast(bf8, u);
}

}  // namespace tile
}  // namespace nystra
