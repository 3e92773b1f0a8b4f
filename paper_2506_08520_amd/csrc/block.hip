// Window-attention block around the PnP-Nystra operator, the structure of
// Sec. 1 for SwinIR / Uformer-style models: the map is cut into w x w windows
// (after a cyclic shift s for shifted windows), Q, K, V = X W_qkv + b per
// token, every (window, head) attends, the heads are concatenated, and
// Y = O W_proj + b goes back to the token's pixel.
//
// Two launches of one MFMA GEMM surround the attention kernels:
//   QKV   rows = tokens in window order, A row r = the pixel of token r in X;
//         the epilogue writes Q, K, V straight into [window][head][N][d_h].
//   PROJ  A row r = token r's d_h-wide slices of O, one per head (the head
//         concatenation is a gather); the epilogue writes Y at the pixel.
// A workgroup computes a 64 x 64 tile of the product over 32-deep chunks of
// the contraction staged in LDS, the next chunk's loads in flight while the
// current one is multiplied; four waves each own a 32 x 32 quarter (2 x 2
// MFMA tiles).  Blocks are mapped so that the column tiles of one row tile
// run on the same XCD and share its L2 for the gathered rows.
#include "internal.hpp"
#include "tile_common.hpp"

namespace nystra {
namespace {

using namespace tile;

constexpr int kBM = 64, kBN = 64, kBK = 32;

struct BlockArgs {
    int64_t rows;                 // tokens, B H W
    int H, W, C, heads, dh, w, N, shift, nwx, nwy;
    int ncols;                    // 3C (QKV) or C (PROJ)
    int rtiles, ctiles;           // tile grid
    const void *a;                // X (QKV) or O (PROJ)
    const void *wt;               // [C][ncols]
    const void *wpk;              // wt packed as the register-resident kernel's LDS tiles
    const void *bias;             // [ncols] or null
    void *out0, *out1, *out2;     // Q, K, V (QKV) or Y (PROJ)
    bool pair;                    // register-resident kernel: store adjacent column pairs
    int64_t ostride;              // register-resident kernel: elements from Q to K and K to V
};

// Flat pixel (b H + y) W + x of token t of window `win`.
__device__ inline int64_t pixel_of(const BlockArgs &a, int64_t win, int t)
{
    const int per = a.nwy * a.nwx;
    const int64_t b = win / per;
    const int wi = int(win - b * per);
    const int wy = wi / a.nwx, wx = wi - wy * a.nwx;
    const int ty = t / a.w, tx = t - ty * a.w;
    int y = wy * a.w + ty + a.shift, x = wx * a.w + tx + a.shift;
    if (y >= a.H)
        y -= a.H;
    if (x >= a.W)
        x -= a.W;
    return (b * a.H + y) * a.W + x;
}

// Block id -> (row tile, column tile), so that consecutive logical tiles (the
// column tiles of one row tile) land on one XCD (ids go round-robin over 8).
__device__ inline void tile_of(const BlockArgs &a, int &rt, int &ct)
{
    const int T = a.rtiles * a.ctiles, q = T / 8, r = T % 8;
    const int b = int(blockIdx.x), x = b % 8, local = b / 8;
    const int L = (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + local;
    rt = L / a.ctiles;
    ct = L - rt * a.ctiles;
}

template <class E>
__device__ inline float ld(const void *p, int64_t i)
{
    return E::load(static_cast<const typename E::T *>(p), i);
}

template <class E, bool PROJ>
__global__ void __launch_bounds__(256) block_gemm_kernel(BlockArgs a)
{
    constexpr bool BF = E::bytes == 2;
    // fp32: A [64][36], B [32][68] floats.  bf16: A [64][40], B^T [64][40] halves.
    constexpr int PA = BF ? kBK + 8 : kBK + 4, PB = BF ? kBK + 8 : kBN + 4;
    __shared__ __align__(16) typename E::T As[kBM * PA];
    __shared__ __align__(16) typename E::T Bs[BF ? kBN * PB : kBK * PB];
    int rt, ct;
    tile_of(a, rt, ct);
    const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, c = lane & 15;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6), wr = wv >> 1, wc = wv & 1;
    const int64_t m0 = int64_t(rt) * kBM;
    const int n0 = ct * kBN;

    // This thread's A row (fixed over the contraction) and B row of a chunk.
    const int arow = tid >> 2, ak = (tid & 3) * 8;
    const int64_t r = m0 + arow;
    const bool rok = r < a.rows;
    const int64_t win = rok ? r / a.N : 0;
    const int t = rok ? int(r - win * a.N) : 0;
    int64_t abase;   // QKV: element offset of the pixel row; PROJ: of head 0's slice
    if constexpr (PROJ)
        abase = (win * a.heads * a.N + t) * int64_t(a.dh);
    else
        abase = pixel_of(a, win, t) * int64_t(a.C);
    const int64_t headstride = int64_t(a.N) * a.dh;
    const int bk = tid >> 3, bn = (tid & 7) * 8;

    float ra[8], rb[8];
    auto fetch = [&](int k0) {
        int k = k0 + ak;
        int hh = 0, dd = 0;
        if constexpr (PROJ) {
            hh = k / a.dh;
            dd = k - hh * a.dh;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float x = 0.f;
            if (rok && k < a.C) {
                if constexpr (PROJ)
                    x = ld<E>(a.a, abase + hh * headstride + dd);
                else
                    x = ld<E>(a.a, abase + k);
            }
            ra[j] = x;
            ++k;
            if constexpr (PROJ) {
                if (++dd == a.dh) {
                    dd = 0;
                    ++hh;
                }
            }
        }
        const int kb = k0 + bk;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int n = n0 + bn + j;
            rb[j] = (kb < a.C && n < a.ncols) ? ld<E>(a.wt, int64_t(kb) * a.ncols + n) : 0.f;
        }
    };
    auto stash = [&]() {
        if constexpr (BF) {
            U16B u;
#pragma unroll
            for (int p = 0; p < 4; ++p)
                u.w[p] = cvt_bf16x2(ra[2 * p], ra[2 * p + 1]);   // exact: bf16 values
            *reinterpret_cast<U16B *>(&As[arow * PA + ak]) = u;
#pragma unroll
            for (int j = 0; j < 8; ++j)
                Bs[(bn + j) * PB + bk] = uint16_t(cvt_bf16x2(rb[j], 0.f));
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                As[arow * PA + ak + j] = ra[j];
                Bs[bk * PB + bn + j] = rb[j];
            }
        }
    };

    f4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
        acc[i][0] = acc[i][1] = f4{0.f, 0.f, 0.f, 0.f};
    fetch(0);
    stash();
    __syncthreads();
    for (int k0 = 0; k0 < a.C; k0 += kBK) {
        const bool more = k0 + kBK < a.C;   // uniform
        if (more)
            fetch(k0 + kBK);
        if constexpr (BF) {
#pragma unroll
            for (int ti = 0; ti < 2; ++ti) {
                const bf8 av = *reinterpret_cast<const bf8 *>(&As[(32 * wr + 16 * ti + c) * PA + 8 * g]);
#pragma unroll
                for (int tj = 0; tj < 2; ++tj) {
                    const bf8 bv =
                        *reinterpret_cast<const bf8 *>(&Bs[(32 * wc + 16 * tj + c) * PB + 8 * g]);
                    acc[ti][tj] = mfma_bf16(av, bv, acc[ti][tj]);
                }
            }
        } else {
#pragma unroll
            for (int s = 0; s < kBK / 4; ++s) {
                float av[2], bv[2];
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    av[i] = As[(32 * wr + 16 * i + c) * PA + 4 * s + g];
                    bv[i] = Bs[(4 * s + g) * PB + 32 * wc + 16 * i + c];
                }
#pragma unroll
                for (int ti = 0; ti < 2; ++ti)
#pragma unroll
                    for (int tj = 0; tj < 2; ++tj)
                        acc[ti][tj] = mfma4(av[ti], bv[tj], acc[ti][tj]);
            }
        }
        __syncthreads();
        if (more) {
            stash();
            __syncthreads();
        }
    }

    // Epilogue: lane (g, c) holds rows 4g + i, column c of each 16 x 16 tile.
#pragma unroll
    for (int tj = 0; tj < 2; ++tj) {
        const int n = n0 + 32 * wc + 16 * tj + c;
        if (n >= a.ncols)
            continue;
        const float bias = a.bias ? ld<E>(a.bias, n) : 0.f;
        int which = 0, hh = 0, dd = n;
        if constexpr (!PROJ) {
            which = n / a.C;
            const int cc = n - which * a.C;
            hh = cc / a.dh;
            dd = cc - hh * a.dh;
        }
        typename E::T *dst = static_cast<typename E::T *>(which == 0 ? a.out0
                                                          : which == 1 ? a.out1 : a.out2);
#pragma unroll
        for (int ti = 0; ti < 2; ++ti)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t row = m0 + 32 * wr + 16 * ti + 4 * g + i;
                if (row >= a.rows)
                    continue;
                const int64_t wn = row / a.N;
                const int tt = int(row - wn * a.N);
                const float v = acc[ti][tj][i] + bias;
                if constexpr (PROJ)
                    E::store(dst, pixel_of(a, wn, tt) * a.C + n, v);
                else
                    E::store(dst, ((wn * a.heads + hh) * a.N + tt) * int64_t(a.dh) + dd, v);
            }
    }
}

// Register-resident variant for C <= 256 (K padded to KP, a multiple of 32).
// Each wave holds its 16 rows of A for the whole contraction in registers, in
// the operand layout of the matrix cores: lane group g takes the contiguous
// quarter k in [g KP/4, (g+1) KP/4), so A is read from memory exactly once.
// The workgroup's eight waves (128 rows) stream W through LDS one 64-column
// tile at a time, double-buffered: the next tile's loads are in flight while
// the current one is multiplied.  W tiles in LDS: fp32 as [k][c][t] (the four
// 16-column tiles' values of column c side by side, one 16-byte read per
// step), bf16 transposed as [n][k] (eight k per 16-byte read).
constexpr int kRkWaves = 8, kRkRows = 16 * kRkWaves;

template <class E, int KP>
struct RkLds {
    static constexpr bool BF = E::bytes == 2;
    static constexpr int PF = 68;            // fp32 [k][c][t]: 64 floats + 4 per k
    static constexpr int PH = KP + 8;        // bf16 [n][k]: halves per column
    static constexpr int tile = BF ? 64 * PH / 2 : KP * PF;   // floats per buffer
    static constexpr int astage = 16 * 8 * (KP / (BF ? 2 : 1) + 8);   // 128 rows, words
    static constexpr int total = 2 * tile > astage ? 2 * tile : astage;
};

// Packs W [C][ncols] into the LDS images of its 64-column tiles, one tile
// after another: bf16 [n][k] with pitch PH (element (k, n0 + n) at n PH + k),
// fp32 [k][PF] with the four 16-column tiles' values of column c at 4c + t
// (element (k, n0 + 16t + c)).  Every slot outside W (k >= C, n >= ncols, the
// pitch padding) is zero.  The second matrix's pieces follow the first's in
// the grid.
struct WPackArgs {
    const void *w0, *w1;   // W_qkv [C][3C], W_proj [C][C]
    uint32_t *d0, *d1;     // their packed images
    int C, words0, words1;
};

template <class E, int KP>
__global__ void __launch_bounds__(256) block_wpack_kernel(WPackArgs p)
{
    // One thread per 16-byte piece of the images (four words).
    using L = RkLds<E, KP>;
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    constexpr int kPieces = L::tile / 4;   // per tile
    const int64_t gi = int64_t(blockIdx.x) * 256 + threadIdx.x;
    const int64_t p0 = p.words0 / 4;
    const bool second = gi >= p0;
    const int64_t pi = second ? gi - p0 : gi;
    if (pi >= (second ? p.words1 / 4 : p0))
        return;
    const int ncols = second ? p.C : 3 * p.C;
    const typename E::T *W = static_cast<const typename E::T *>(second ? p.w1 : p.w0);
    const int ct = int(pi / kPieces), r = int(pi - int64_t(ct) * kPieces), n0 = 64 * ct;
    // Branch-free: every load reads an in-bounds element (indices clamped) and
    // a select zeroes the slots outside W, so a thread's loads issue together.
    auto elem = [&](int k, int n) -> uint32_t {
        const bool ok = k < p.C && n < ncols;
        const int64_t i = int64_t(k < p.C ? k : p.C - 1) * ncols + (n < ncols ? n : ncols - 1);
        uint32_t x;
        if constexpr (E::bytes == 2)
            x = uint32_t(reinterpret_cast<const uint16_t *>(W)[i]);
        else
            x = __float_as_uint(W[i]);
        return ok ? x : 0u;
    };
    u32x4 out;
    int dst;   // piece index within the tile image
    if constexpr (E::bytes == 2) {
        // column n = r mod 64 (consecutive threads: consecutive columns of
        // eight rows of W), halves k0 .. k0 + 7 of its image row
        const int n = r & 63, k0 = 8 * (r >> 6);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int k = k0 + 2 * e;
            out[e] = elem(k, n0 + n) | (elem(k + 1, n0 + n) << 16);   // zero from k = C on
        }
        dst = (n * L::PH + k0) / 8;
    } else {
        // row k, column c: the four 16-column tiles' values (slot 16 of a row
        // is the pitch padding)
        const int k = r / (L::PF / 4), c = r - k * (L::PF / 4);
#pragma unroll
        for (int t = 0; t < 4; ++t)
            out[t] = c < 16 ? elem(k, n0 + 16 * t + c) : 0u;
        dst = r;
    }
    reinterpret_cast<u32x4 *>(second ? p.d1 : p.d0)[int64_t(ct) * kPieces + dst] = out;
}

// Words per batch of the A stage: the largest divisor of n up to 16.
constexpr int stage_batch(int n)
{
    for (int b = 16; b > 1; --b)
        if (n % b == 0)
            return b;
    return 1;
}

template <class E, bool PROJ, int KP>
__global__ void __launch_bounds__(64 * kRkWaves) block_gemm_rk_kernel(BlockArgs a)
{
    constexpr bool BF = E::bytes == 2;
    using L = RkLds<E, KP>;
    constexpr int KQ = KP / 4;               // contraction slots per lane group
    __shared__ __align__(16) float lds_all[L::total];
    auto wbuf = [&](int b) { return lds_all + b * L::tile; };
    const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, c = lane & 15;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t m0 = int64_t(blockIdx.x) * kRkRows;

    // ---- A: the workgroup's 128 rows are staged in LDS with coalesced 4-byte
    // loads (lanes take consecutive words of a row; bf16 words hold two
    // elements), then each lane copies its operand slots -- row 16 wv + c,
    // k = g KQ + s -- into registers.  The stage shares LDS with the W tiles.
    constexpr int EPW = BF ? 2 : 1;              // elements per 4-byte word
    constexpr int AWL = KP / EPW;                // words per staged row
    constexpr int AP = AWL + 8;                  // row pitch (words; + 8: fewer bank conflicts
                                                 // than + 4 in the operand reads)
    __shared__ int rowbase[kRkRows];             // element offset of row r (-1: none)
    __shared__ int colofs[AWL];                  // element offset of word w in a row
    float *astage = lds_all;
    if (tid < kRkRows) {
        const int64_t row = m0 + tid;
        int base = -1;
        if (row < a.rows) {
            const int wn = int(row / a.N), tt = int(row - int64_t(wn) * a.N);
            base = int(PROJ ? (int64_t(wn) * a.heads * a.N + tt) * a.dh
                            : pixel_of(a, wn, tt) * a.C);
        }
        rowbase[tid] = base;
    }
    for (int w = tid; w < AWL; w += 64 * kRkWaves) {
        const int k = w * EPW;
        int off = k;
        if constexpr (PROJ) {
            const int hh = k / a.dh;
            off = hh * a.N * a.dh + (k - hh * a.dh);
        }
        colofs[w] = k < a.C ? off : -1;
    }
    // ---- W tiles: the packed image of each 64-column tile (block_wpack_kernel
    // lays it out exactly as the LDS tile below, padding included) is copied
    // global -> registers -> LDS in 16-byte pieces, consecutive lanes taking
    // consecutive pieces: coalesced loads, conflict-free stores, no index
    // arithmetic per element.
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    constexpr int kPieces = L::tile / 4;   // 16-byte pieces of a tile image
    constexpr int kPer = (kPieces + 64 * kRkWaves - 1) / (64 * kRkWaves);
    u32x4 wr[kPer];
    const int nct = (a.ncols + 63) / 64;
    const u32x4 *wsrc = static_cast<const u32x4 *>(a.wpk);
    auto wfetch = [&](int ct) {
        const u32x4 *src = wsrc + int64_t(ct) * kPieces;
#pragma unroll
        for (int j = 0; j < kPer; ++j) {   // past the image: re-read its last piece
            const int idx = tid + j * 64 * kRkWaves;
            wr[j] = src[idx < kPieces ? idx : kPieces - 1];
        }
    };
    auto wstash = [&](int buf) {
        u32x4 *dst = reinterpret_cast<u32x4 *>(wbuf(buf));
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
            const int idx = tid + j * 64 * kRkWaves;
            if (kPer * 64 * kRkWaves == kPieces || idx < kPieces)
                dst[idx] = wr[j];
        }
    };
    // Workgroups start at different column tiles, so that at any moment they
    // read different tiles of W instead of all hitting the same L2 lines.
    const int start = int(blockIdx.x % unsigned(nct));
    auto phys = [&](int i) { return i + start < nct ? i + start : i + start - nct; };
    // The first W tile and the bias are requested now, their latency hidden
    // behind the A stage; the bias of every column is staged in LDS once (a
    // global load in the epilogue would wait behind the next tile's W pieces
    // in flight).
    wfetch(phys(0));
    __shared__ float colbias[3 * 256];
    constexpr int kBiasPer = (3 * 256 + 64 * kRkWaves - 1) / (64 * kRkWaves);
    float bz[kBiasPer];
#pragma unroll
    for (int j = 0; j < kBiasPer; ++j) {
        const int n = tid + j * 64 * kRkWaves;
        const int nc = n < a.ncols ? n : a.ncols - 1;
        bz[j] = a.bias ? ld<E>(a.bias, nc) : 0.f;
    }
    __syncthreads();
    {
        // Each thread copies kPerT words, in batches whose loads are all in
        // flight before the first is waited for (a loop of load, wait, store
        // would chain kPerT memory round trips).
        constexpr int kPerT = kRkRows * AWL / (64 * kRkWaves);
        constexpr int kBatch = stage_batch(kPerT);
        static_assert(kPerT * 64 * kRkWaves == kRkRows * AWL, "whole words per thread");
        const uint32_t *src = static_cast<const uint32_t *>(a.a);
        uint32_t *dst = reinterpret_cast<uint32_t *>(astage);
        for (int b0 = 0; b0 < kPerT; b0 += kBatch) {
            uint32_t x[kBatch];
            int at[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int j = tid + (b0 + u) * 64 * kRkWaves;
                const int row = j / AWL, w = j - row * AWL;
                const int rb = rowbase[row], co = colofs[w];
                const bool ok = rb >= 0 && co >= 0;
                const int e = ok ? rb + co : 0;
                x[u] = src[BF ? e >> 1 : e];
                at[u] = ok ? row * AP + w : -1;
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int j = tid + (b0 + u) * 64 * kRkWaves;
                const int row = j / AWL, w = j - row * AWL;
                dst[row * AP + w] = at[u] >= 0 ? x[u] : 0u;
            }
        }
    }
    __syncthreads();
    float av[BF ? 1 : KQ];
    bf8 ab[BF ? KQ / 8 : 1];
    {
        const float *arow = astage + (16 * wv + c) * AP;
        if constexpr (BF) {
#pragma unroll
            for (int s = 0; s < KQ / 8; ++s)
                ab[s] = *reinterpret_cast<const bf8 *>(arow + (g * KQ + 8 * s) / 2);
        } else {
#pragma unroll
            for (int s = 0; s < KQ; s += 4) {
                const f4 v = *reinterpret_cast<const f4 *>(arow + g * KQ + s);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    av[s + e] = v[e];
            }
        }
    }
    __syncthreads();   // the stage becomes the W tiles

    // Column part of the destination for the 64 columns of the current tile,
    // from out0: (QKV) output tensor `which` at which * ostride, head h,
    // feature f -> h N d_h + f; (PROJ) the column.
    __shared__ uint32_t coltab[2][64];
    auto cfill = [&](int ct, int buf) {
        if (tid < 64) {
            const int n = 64 * ct + tid;
            int which = 0, col = n;
            if constexpr (!PROJ) {
                which = n / a.C;
                const int cc = n - which * a.C;
                const int hh = cc / a.dh;
                col = hh * a.N * a.dh + (cc - hh * a.dh);
            }
            coltab[buf][tid] = uint32_t(which * a.ostride + col);
        }
    };

    // Row part of the destination of this lane's output rows 4g + i: QKV
    // (window wn, token tt) -> wn N C + tt d_h; PROJ -> pixel C.  Offsets are
    // unsigned 32-bit (tensors under 2^31 elements); rows past the end are
    // not stored.
    uint32_t rowoff[4];
    bool rowok[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = int(m0) + 16 * wv + 4 * g + i;   // rows < 2^31
        rowok[i] = row < a.rows;
        const int rr = rowok[i] ? row : 0;
        const int wn = rr / a.N, tt = rr - wn * a.N;
        rowoff[i] = uint32_t(PROJ ? pixel_of(a, wn, tt) * a.C
                                  : int64_t(wn) * a.N * a.C + int64_t(tt) * a.dh);
    }

#pragma unroll
    for (int j = 0; j < kBiasPer; ++j) {
        const int n = tid + j * 64 * kRkWaves;
        if (n < a.ncols)
            colbias[n] = bz[j];
    }
    wstash(0);
    cfill(phys(0), 0);
    __syncthreads();
    for (int it = 0; it < nct; ++it) {
        const int ct = phys(it);
        const bool more = it + 1 < nct;   // uniform
        if (more)
            wfetch(phys(it + 1));
        const float *wt = wbuf(it & 1);
        f4 acc[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
            acc[q] = f4{0.f, 0.f, 0.f, 0.f};
        if constexpr (BF) {
            const uint16_t *h = reinterpret_cast<const uint16_t *>(wt);
#pragma unroll
            for (int s = 0; s < KQ / 8; ++s)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const bf8 bv = *reinterpret_cast<const bf8 *>(
                        &h[(16 * q + c) * L::PH + g * KQ + 8 * s]);
                    acc[q] = mfma_bf16(ab[s], bv, acc[q]);
                }
        } else {
#pragma unroll
            for (int s = 0; s < KQ; ++s) {
                const f4 bv = *reinterpret_cast<const f4 *>(&wt[(g * KQ + s) * L::PF + 4 * c]);
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    acc[q] = mfma4(av[s], bv[q], acc[q]);
            }
        }
        // The next tile goes to the idle buffer before this tile's stores are
        // issued: the wait for its loads counts every earlier vector memory
        // operation, stores included, so stashing after the stores would
        // wait for their completion on every tile.
        if (more) {
            wstash((it + 1) & 1);
            cfill(phys(it + 1), (it + 1) & 1);
        }
        // Epilogue: lane (g, c) holds rows 4g + i of the wave's 16, column c of tile q;
        // destination = row part (per lane, computed once) + column part (table).
        // With a.pair, lanes c and c ^ 1 swap one value per two rows so that the
        // even lane holds columns (c, c + 1) of row 4g + 2p and the odd lane
        // those of row 4g + 2p + 1: one 4-byte (bf16) or 8-byte (fp32) store per
        // two outputs.  Pairs never straddle a head or Q/K/V (d_h and C even).
        if (a.pair) {
            const bool odd = c & 1;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int n = 64 * ct + 16 * q + c;   // n and n ^ 1 lie on one side of ncols
                if (n >= a.ncols)
                    continue;
                const float bias = colbias[n];
                const int cp = (16 * q + c) & ~1;
                const uint32_t col = coltab[it & 1][cp];
                typename E::T *dst = static_cast<typename E::T *>(a.out0);
#pragma unroll
                for (int pp = 0; pp < 2; ++pp) {
                    const float v0 = acc[q][2 * pp] + bias, v1 = acc[q][2 * pp + 1] + bias;
                    const float recv = dpp_xor1(odd ? v0 : v1);
                    const float lo = odd ? recv : v0, hi = odd ? v1 : recv;
                    const int i = 2 * pp + (odd ? 1 : 0);
                    if (rowok[i]) {
                        if constexpr (BF)
                            *reinterpret_cast<uint32_t *>(dst + (rowoff[i] + col)) =
                                cvt_bf16x2(lo, hi);   // RNE
                        else
                            *reinterpret_cast<float2 *>(dst + (rowoff[i] + col)) =
                                make_float2(lo, hi);
                    }
                }
            }
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int n = 64 * ct + 16 * q + c;
                if (n >= a.ncols)
                    continue;
                const float bias = colbias[n];
                const uint32_t col = coltab[it & 1][16 * q + c];
                typename E::T *dst = static_cast<typename E::T *>(a.out0);
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (rowok[i]) {
                        const float v = acc[q][i] + bias;
                        if constexpr (BF)
                            dst[rowoff[i] + col] = uint16_t(cvt_bf16x2(v, 0.f));   // RNE
                        else
                            dst[rowoff[i] + col] = v;
                    }
            }
        }
        __syncthreads();
    }
}

template <class E, bool PROJ, int KP>
void launch_rk(const BlockArgs &a, hipStream_t stream)
{
    const unsigned blocks = unsigned((a.rows + kRkRows - 1) / kRkRows);
    hipLaunchKernelGGL((block_gemm_rk_kernel<E, PROJ, KP>), dim3(blocks), dim3(64 * kRkWaves), 0,
                       stream, a);
}

template <class E, bool PROJ>
bool try_rk(const BlockArgs &a, hipStream_t stream)
{
    if (!a.wpk)
        return false;   // the weights were not packed (C > 256)
    if (a.rows * int64_t(a.C) >= (int64_t(1) << 31) ||
        int64_t(a.C) * a.ncols >= (int64_t(1) << 31))
        return false;   // 32-bit element offsets
    if ((a.rows + kRkRows - 1) / kRkRows * 64 * kRkWaves >= (int64_t(1) << 32))
        return false;   // fewer than 2^32 work-items in the grid
    // A as 4-byte words: bf16 needs an even C, and in PROJ an even d_h (a word
    // never straddles two heads); the A base 4-byte aligned
    if (uintptr_t(a.a) % 4 != 0 || (E::bytes == 2 && (a.C % 2 != 0 || (PROJ && a.dh % 2 != 0))))
        return false;
    // One output base: Q, K, V at a uniform element stride from out0, every
    // offset under 2^32 elements.
    BlockArgs b = a;
    b.ostride = 0;
    if constexpr (!PROJ) {
        const int64_t s1 = static_cast<const char *>(a.out1) - static_cast<const char *>(a.out0);
        const int64_t s2 = static_cast<const char *>(a.out2) - static_cast<const char *>(a.out1);
        if (s1 != s2 || s1 < 0 || s1 % E::bytes != 0)
            return false;
        b.ostride = s1 / E::bytes;
        if (3 * b.ostride >= (int64_t(1) << 32) || b.ostride < a.rows * int64_t(a.C))
            return false;
    }
    // paired column stores: even widths, outputs aligned to two elements
    const uintptr_t al = 2 * E::bytes;
    b.pair = a.ncols % 2 == 0 && a.dh % 2 == 0 && uintptr_t(a.out0) % al == 0 &&
             (PROJ || (uintptr_t(a.out1) % al == 0 && uintptr_t(a.out2) % al == 0));
    if (a.C <= 32)
        launch_rk<E, PROJ, 32>(b, stream);
    else if (a.C <= 64)
        launch_rk<E, PROJ, 64>(b, stream);
    else if (a.C <= 128)
        launch_rk<E, PROJ, 128>(b, stream);
    else if (a.C <= 192)
        launch_rk<E, PROJ, 192>(b, stream);
    else if (a.C <= 256)
        launch_rk<E, PROJ, 256>(b, stream);
    else
        return false;
    return true;
}

template <class E, bool PROJ>
void launch_gemm(const BlockArgs &a, hipStream_t stream)
{
    if (try_rk<E, PROJ>(a, stream))
        return;
    const unsigned blocks = unsigned(a.rtiles) * unsigned(a.ctiles);
    hipLaunchKernelGGL((block_gemm_kernel<E, PROJ>), dim3(blocks), dim3(256), 0, stream, a);
}

}  // namespace

bool block_gemm_supported(int64_t rows, int C)
{
    const int64_t rt = (rows + kBM - 1) / kBM, ct = (3 * int64_t(C) + kBN - 1) / kBN;
    return rt * ct * 256 < (int64_t(1) << 32);
}

// Contraction length of the register-resident kernel for C (0: not used).
static int rk_kp(int C)
{
    return C <= 32 ? 32 : C <= 64 ? 64 : C <= 128 ? 128 : C <= 192 ? 192 : C <= 256 ? 256 : 0;
}

template <class E, int KP>
size_t wpack_words(int ncols)
{
    return size_t((ncols + 63) / 64) * RkLds<E, KP>::tile;
}

template <class E>
size_t wpack_words_e(int C, int ncols)
{
    switch (rk_kp(C)) {
    case 32: return wpack_words<E, 32>(ncols);
    case 64: return wpack_words<E, 64>(ncols);
    case 128: return wpack_words<E, 128>(ncols);
    case 192: return wpack_words<E, 192>(ncols);
    case 256: return wpack_words<E, 256>(ncols);
    default: return 0;
    }
}

size_t block_wpack_bytes(int C, int ncols, int dtype)
{
    return 4 * (dtype == 0 ? wpack_words_e<F32>(C, ncols) : wpack_words_e<BF16>(C, ncols));
}

template <class E, int KP>
void launch_wpack_k(const WPackArgs &p, hipStream_t stream)
{
    const int64_t pieces = (int64_t(p.words0) + p.words1) / 4;   // tiles are whole pieces
    hipLaunchKernelGGL((block_wpack_kernel<E, KP>), dim3(unsigned((pieces + 255) / 256)),
                       dim3(256), 0, stream, p);
}

template <class E>
void launch_wpack_e(const WPackArgs &p, hipStream_t stream)
{
    switch (rk_kp(p.C)) {
    case 32: launch_wpack_k<E, 32>(p, stream); break;
    case 64: launch_wpack_k<E, 64>(p, stream); break;
    case 128: launch_wpack_k<E, 128>(p, stream); break;
    case 192: launch_wpack_k<E, 192>(p, stream); break;
    default: launch_wpack_k<E, 256>(p, stream); break;
    }
}

hipError_t launch_block_wpack(const void *wqkv, const void *wproj, int C, int dtype, void *pk_qkv,
                              void *pk_proj, hipStream_t stream)
{
    WPackArgs p;
    p.w0 = wqkv;
    p.w1 = wproj;
    p.d0 = static_cast<uint32_t *>(pk_qkv);
    p.d1 = static_cast<uint32_t *>(pk_proj);
    p.C = C;
    p.words0 = int(block_wpack_bytes(C, 3 * C, dtype) / 4);
    p.words1 = int(block_wpack_bytes(C, C, dtype) / 4);
    if (dtype == 0)
        launch_wpack_e<F32>(p, stream);
    else
        launch_wpack_e<BF16>(p, stream);
    return hipGetLastError();
}

hipError_t launch_block_gemm(const BlockGemm &g, hipStream_t stream)
{
    BlockArgs a;
    a.rows = g.rows;
    a.H = g.H;
    a.W = g.W;
    a.C = g.C;
    a.heads = g.heads;
    a.dh = g.C / g.heads;
    a.w = g.w;
    a.N = g.w * g.w;
    a.shift = g.shift;
    a.nwx = g.W / g.w;
    a.nwy = g.H / g.w;
    a.ncols = g.proj ? g.C : 3 * g.C;
    a.rtiles = int((g.rows + kBM - 1) / kBM);
    a.ctiles = (a.ncols + kBN - 1) / kBN;
    a.a = g.a;
    a.wt = g.wt;
    a.wpk = g.wpk;
    a.bias = g.bias;
    a.out0 = g.out0;
    a.out1 = g.out1;
    a.out2 = g.out2;
    a.pair = false;
    a.ostride = 0;
    if (g.dtype == 0)
        g.proj ? launch_gemm<F32, true>(a, stream) : launch_gemm<F32, false>(a, stream);
    else
        g.proj ? launch_gemm<BF16, true>(a, stream) : launch_gemm<BF16, false>(a, stream);
    return hipGetLastError();
}

}  // namespace nystra
