// Internal interface between the C-ABI layer (forge_api.cpp) and the HIP kernels
// (forge_kernels.hip).  Not installed; callers use include/forge.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace forge_impl {

// Scalars of one optimizer step, precomputed on the host in fp64 and rounded to fp32.  For
// AdamW (Algorithm 1: the state recurrences and the bias-corrected, decoupled update) the
// first eight are used; the other rules of the family table read the fields named in their
// element functions (forge_kernels.hip).
struct Hyper {
    float b1, c1;          // beta1, 1 - beta1 (AdamW); the first decay of the other rules
    float b2, c2;          // beta2, 1 - beta2
    float lr_bc1;          // lr / (1 - beta1^t)
    float inv_sqrt_bc2;    // 1 / sqrt(1 - beta2^t)
    float eps;
    float wdf;             // 1 - lr * weight_decay (decoupled decay)
    float lr;              // learning rate (Adagrad: lr / (1 + (t-1) lr_decay))
    float wd;              // weight decay added to the gradient (coupled decay)
    float ka, kb;          // NAdam, RAdam: step coefficients of their two update terms
};

// Everything a launch needs; passed by value as the kernel argument.
struct Args {
    const uint16_t *X;     // bf16 [T, d_in]
    const uint16_t *dY;    // bf16 [T, d_out]
    uint16_t *W;           // bf16 [d_out, d_in]
    void *m, *v;           // moments, storage per moment dtype
    float *ms, *vs;        // int8 block scales: [ceil(d_out/256), d_in], or [d_out, ceil(d_in/64)]
    void *G;               // materialised gradient (two-kernel path only)
    float *wr;             // fp8 weights: amax ring of W [AMAX_SLOTS]
    int T, d_in, d_out;
    int slot;              // fp8 tensors: step % AMAX_SLOTS
    int tiles_p, tiles_q;  // tile grid (along d_out, along d_in)
    int group_p;           // raster group height in tiles (L2 reuse of operand slabs)
    Hyper h;
};

// Up to this many independent matrices share one fused launch (forge_linear_step_grouped).
constexpr int MAX_GROUP = 8;

// A launch over several matrices: their tiles are concatenated, matrix i owning global
// tiles [start[i], start[i+1]).  Passed by value as the kernel argument (about 1 KB).
struct GroupArgs {
    Args a[MAX_GROUP];
    int start[MAX_GROUP + 1];
    int n;
};

// One term dY_s W_s of the input gradient (forge_dx.hip): dY_s bf16 [T, d_out],
// W_s bf16 [d_out, d_in]; d_out > 0.
struct DxSeg {
    const uint16_t *dY;
    const uint16_t *W;
    int d_out;
};

// A launch of the input-gradient GEMM dX = sum_s dY_s W_s (kernel argument).
struct DxArgs {
    DxSeg s[MAX_GROUP];
    int n;                 // segments
    int nch;               // K chunks over all segments
    uint16_t *dX;          // bf16 [T, d_in]
    int T, d_in;
    int tiles_t, tiles_q;  // tile grid (along T, along d_in)
    int group_t;           // raster group height in tiles
};

// Moment storage: fp32, bf16, int8 with one scale per 256 rows of a column (sqrt(v)
// stored), int8 with one scale per 64 consecutive elements of a row (v stored), fp8 E4M3
// with one delayed scale per tensor (m and sqrt(v) stored).
enum MomentKind { MK_F32 = 0, MK_BF16 = 1, MK_I8 = 2, MK_I8R64 = 3, MK_FP8 = 4 };
// fp8 tensors keep a ring of AMAX_SLOTS amax values; step t writes slot t % 4.
constexpr int AMAX_SLOTS = 4;
constexpr int I8_ROW_BLOCK = 64;
// Tile epilogues of the fused kernel: the update rules (each a per-element function of G,
// W and the rule's state), and the store-G control.
enum EpiKind {
    EPI_ADAMW = 0, EPI_STORE_BF16 = 1, EPI_STORE_F32 = 2,
    EPI_SGD = 3, EPI_SGDM = 4, EPI_ADAGRAD = 5, EPI_RMSPROP = 6, EPI_LION = 7,
    EPI_NADAM = 8, EPI_RADAM = 9, EPI_ADAMAX = 10, EPI_MUON = 11,
    EPI_ADAMW_WFP8 = 12,   // AdamW with W stored as fp8 E4M3 (per-tensor delayed scale)
    EPI_COUNT = 13
};

struct TileShape { int rows, cols, tokens; };

// Tile geometry used for a moment kind (fused step and stand-alone optimizer alike).
TileShape tile_shape(int moment_kind);

// Launchers; they return the hipError_t of the launch.
hipError_t launch_fused(const Args &a, int moment_kind, hipStream_t stream);
// n matrices (1 <= n <= MAX_GROUP, none empty) in one launch; all share T and the step.
hipError_t launch_fused_group(const Args *a, int n, int moment_kind, hipStream_t stream);
// The fused step with update rule `epi` (any EpiKind but the store-G ones) on fp32 or bf16
// state: n matrices (1 <= n <= MAX_GROUP, none empty) in one launch.
hipError_t launch_fused_rule(const Args *a, int n, int epi, int moment_kind, hipStream_t stream);
// AdamW with fp8 weights (and bf16 or fp8 moments): n matrices in one launch.
hipError_t launch_fused_wfp8(const Args *a, int n, int moment_kind, hipStream_t stream);
hipError_t launch_wgrad(const Args &a, int grad_f32, hipStream_t stream);
hipError_t launch_adamw(const Args &a, int moment_kind, int grad_f32, hipStream_t stream);
// dX = sum of dY_s W_s over n segments (0 <= n <= MAX_GROUP, none with d_out == 0; n == 0
// writes zeros).  No launch when T == 0 or d_in == 0.
hipError_t launch_dx(const DxSeg *s, int n, uint16_t *dX, int T, int d_in, hipStream_t stream);

// Compute units of the current device (cached per device ordinal; 256 if unknown).
int device_cu_count();

// The fixed device buffer of forge_linear_step_unfused_noalloc (forge_scratch.hip): its
// size, and its address on the current device (looked up once per device ordinal below
// MAX_DEVICES).
constexpr int64_t SCRATCH_BYTES = int64_t(64) << 20;
constexpr int MAX_DEVICES = 64;
hipError_t scratch_address(void **out);

}  // namespace forge_impl
