// Internal interfaces between the C-ABI dispatch layer and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nystra {

// Pooling grid of Step 1 (Sec. 2.2).  Token t = r * cols + c of the window
// averages into landmark (r / pr) * gc + (c / pc).  The 1-D mode is the same
// grid with a single row of N tokens.
struct Geometry {
    int rows, cols;  // token grid
    int pr, pc;      // patch rows / columns
    int gc;          // patches per grid row
};

// Returns false when (N, m, mode) has no pooling grid.
bool make_geometry(int N, int m, int mode, Geometry *g);

struct Problem {
    const void *q, *k, *v;
    void *o;
    int64_t units;   // n_windows * heads
    int N, d, m;
    int iters;
    int dtype;       // 0 = fp32, 1 = bf16
    float scale;     // resolved logit scale (> 0)
    Geometry geo;
};

// Each launcher enqueues on `stream` and returns hipGetLastError().
hipError_t launch_generic_forward(const Problem &p, hipStream_t stream);
hipError_t launch_landmark_pool(const Problem &p, float *qbar, float *kbar, int32_t *map,
                                hipStream_t stream);
hipError_t launch_exact(const Problem &p, hipStream_t stream);

// MFMA-tiled Nystrom kernels.  tiled_supported() is a host-side test of
// whether a shape has a tiled kernel; launch_tiled_forward() requires it and
// picks the one-wave kernel for windows of at most 64 tokens and 16
// landmarks, the multi-wave kernel otherwise.
bool tiled_supported(const Problem &p);
hipError_t launch_tiled_forward(const Problem &p, hipStream_t stream);
bool tiled_large_supported(const Problem &p);
hipError_t launch_tiled_large(const Problem &p, hipStream_t stream);

// Token-split kernels over a caller-provided workspace (global attention).
// split_supported() is a host-side test of the shape and pointers;
// split_workspace_bytes() is the workspace size launch_split() needs, which
// must be 256-byte aligned.
bool split_supported(const Problem &p);
size_t split_workspace_bytes(const Problem &p);
hipError_t launch_split(const Problem &p, void *workspace, hipStream_t stream);

// Projection GEMMs of the window-attention block.  QKV (proj = false): A rows
// are the pixels of X in window order, outputs go to Q, K, V (out0..2) in
// [window][head][N][d_h].  PROJ: A rows gather the heads of O, outputs go to
// the pixels of Y (out0).  Weights are [C][3C] or [C][C]; bias may be null.
// wpk: the weights packed by launch_block_wpack (C <= 256), or null.
struct BlockGemm {
    int64_t rows;     // B H W
    int H, W, C, heads, w, shift, dtype;
    bool proj;
    const void *a, *wt, *bias, *wpk;
    void *out0, *out1, *out2;
};
bool block_gemm_supported(int64_t rows, int C);
hipError_t launch_block_gemm(const BlockGemm &g, hipStream_t stream);
// Bytes of the packed image of a [C][ncols] weight matrix (0 when C > 256:
// the GEMM then reads the weights directly), and one launch packing W_qkv
// ([C][3C]) into pk_qkv and W_proj ([C][C]) into pk_proj.
size_t block_wpack_bytes(int C, int ncols, int dtype);
hipError_t launch_block_wpack(const void *wqkv, const void *wproj, int C, int dtype, void *pk_qkv,
                              void *pk_proj, hipStream_t stream);

// Head widths with a tiled instantiation: the multiples of 4 from 8 to 32
// (Dehazeformer's 12 and 16, Uformer's 32) and SwinIR's 30.
inline bool tiled_width(int d) { return d >= 8 && d <= 32 && (d % 4 == 0 || d == 30); }

}  // namespace nystra
