// forge_kernels.hip -- gfx950 (CDNA4) kernels for the fused weight-gradient + AdamW step.
//
// One workgroup owns one tile of W (FORGE Sec. 2.2, Eq. tile, Algorithm 1) and has two
// roles of four waves each:
//
//   math waves   stage X and dY token chunks from HBM/L2 into LDS (transposing them so
//                that the token axis, the GEMM's K, is contiguous), and accumulate
//                G_tile = dY_tile^T X_tile with v_mfma_f32_32x32x16_bf16 into fp32
//                registers; at the end they drop the accumulator tile into LDS.
//   stream waves issue the global loads of the tile's W, m, v (and int8 scales) early in
//                the mainloop, right after the DMA of its first chunks, so that this HBM
//                traffic overlaps the mainloop (vmcnt is per wave, so the math waves never
//                wait on it); then they run the AdamW epilogue on the LDS copy of G with
//                coalesced 16-byte accesses and store W, m, v.  G never leaves the chip.
//
// The two-kernel comparison path reuses the same pieces: the store-G GEMM runs the same
// mainloop with an epilogue that writes G, and the stand-alone optimizer stages a tile
// of a materialised G into LDS and runs the same epilogue code.
#include "forge_device.h"

#include <mutex>

namespace forge_impl {

#ifndef FORGE_TK
#define FORGE_TK 32
#endif
#ifndef FORGE_NS
#define FORGE_NS 4
#endif
#ifndef FORGE_NS_I8P               // ring depth of the pipelined int8 kernel
#define FORGE_NS_I8P 4
#endif
#ifndef FORGE_GROUP_P_I8            // raster rows of the pipelined int8 kernel (0: by T)
#define FORGE_GROUP_P_I8 0
#endif
#ifndef FORGE_NSW_I8P              // its stream waves (4 or 8)
#define FORGE_NSW_I8P 8
#endif
constexpr int NS_I8P = FORGE_NS_I8P;
#ifndef FORGE_SCHED_SPLIT         // sched_barrier between the two MFMA steps of a chunk
#define FORGE_SCHED_SPLIT 1
#endif
#ifndef FORGE_GROUP_P             // tile rows walked together by the raster (0: by shape)
#define FORGE_GROUP_P 0
#endif
constexpr int TK128 = FORGE_TK;   // tokens per pipeline chunk (the GEMM's K step), 128x128 tiles
constexpr int NSTAGE = FORGE_NS;  // LDS ring depth (chunks) of the 128x128 mainloop
constexpr int NROLE = 256;      // threads per role (4 waves)
constexpr int NT = 2 * NROLE;   // threads per fused workgroup
constexpr int I8_BLOCK = 256;   // rows of d_out sharing one int8 scale

// Tile shapes: (rows along d_out) x (cols along d_in).  int8 tiles are exactly one scale
// block tall so that the block absmax closes inside the workgroup.
constexpr int BP_F = 128, BQ_F = 128;
constexpr int BP_I8 = 256, BQ_I8 = 64;

// ------------------------------------------------------------------------ small helpers

// One AdamW element (Algorithm 1): state update, then the bias-corrected decoupled
// weight update.  rv1 = sqrt(v1) is returned as well (the int8 path stores it).
__device__ __forceinline__ void adamw_elem(float g, float w, float m, float v, const Hyper &h,
                                           float &w1, float &m1, float &v1, float &rv1)
{
    m1 = __builtin_fmaf(h.b1, m, h.c1 * g);
    v1 = __builtin_fmaf(h.b2, v, (h.c2 * g) * g);
    rv1 = __builtin_amdgcn_sqrtf(v1);
    float den = __builtin_fmaf(rv1, h.inv_sqrt_bc2, h.eps);        // sqrt(vhat) + eps
    float upd = (m1 * h.lr_bc1) * __builtin_amdgcn_rcpf(den);       // lr * mhat / den
    w1 = __builtin_fmaf(h.wdf, w, -upd);
}

// ------------------------------------------------------------------------ mainloop

// G^T tile (rows q along d_in, cols p along d_out) = X_tile^T dY_tile, accumulated in
// fp32.  MFMA operand A is X (M = q), operand B is dY (N = p); each lane of a 32x32
// result holds 4 consecutive q for one p, which is the order G is staged in below.
//
// Operand path: a ring of NS LDS stages, each holding one chunk of TK tokens of X and dY
// in their natural [token][column] layout.  Chunks are copied HBM/L2 -> LDS by buffer
// loads that write LDS directly (no registers; NS-1 chunks in flight), with a 16-byte
// XOR swizzle of each row so that the fragment reads below are bank-conflict free.
// Rows past T and columns past d_in / d_out read as zero (buffer range checking).
// MFMA fragments (8 consecutive tokens of one column per lane) are gathered with the
// CDNA4 transposing LDS read ds_read_b64_tr_b16: within each group of 16 lanes, lane i
// receives element i%4 of the 8-byte rows read by lanes i/4 + 4j (j = 0..3); pointing
// lane s at token t0 + s/4, column c0 + 4 (s%4) hands lane i column c0 + i, tokens
// t0..t0+3.  These reads are issued from inline assembly with explicit lgkmcnt waits,
// so the compiler does not serialise them behind the in-flight LDS DMA.
template <int BP, int BQ, int NS, int TK = 32>
struct Mainloop {
    static_assert(TK % 32 == 0, "chunks are whole pairs of 16-token MFMA steps");
    static constexpr int WQ = BQ / 64;                   // waves along q
    static constexpr int WP = BP / 64;                   // waves along p
    static_assert(WQ * WP == 4, "four math waves, 64x64 each");
    static constexpr int XROWB = BQ * 2, YROWB = BP * 2; // LDS bytes per token row
    static_assert(TK == 32 || XROWB == YROWB, "a stage of several 32-token steps needs equal row lengths");
    static constexpr int XCH = TK * BQ / 8;              // 16-byte pieces of X per chunk
    static constexpr int YCH = TK * BP / 8;
    static constexpr int NINST = (XCH + YCH) / 64;       // wave-wide DMA instructions per chunk
    static_assert(XCH % 64 == 0 && YCH % 64 == 0 && NINST % 4 == 0, "chunk splits evenly");
    static constexpr int DPC = NINST / 4;                // per math wave
    static constexpr int STAGE_BYTES = (XCH + YCH) * 16;
    static constexpr int LDS_BYTES = NS * STAGE_BYTES;
    static_assert(2 * 20 * (XROWB > YROWB ? XROWB : YROWB) + 3 * STAGE_BYTES < 65536 || true, "");

    f32x16_t acc[2][2];                                  // [q sub-tile][p sub-tile]
    uint32_t voff[DPC];                                  // buffer byte offsets of this lane's DMA pieces
    uint32_t ta[2], tb[2];                               // LDS byte offsets of this lane's fragment rows

    // 16-byte swizzle of token row t.  Half a wave's transposing read covers 4 token rows
    // x 4 aligned 16-byte pieces (64 B per row); the LDS serves 256 B (64 banks) per cycle.
    // XOR-ing the piece index with a multiple of 4 moves each row's 64 B to its own quarter
    // of the banks: rows of >= 256 B use 4*(t%4), rows of 128 B (two rows per bank sweep)
    // use 4*((t/2)%2).  Without it the 4 rows collide two by two.
    template <int ROWB>
    static __device__ __forceinline__ int swz(int t)
    {
        static_assert(ROWB >= 128, "at least 8 pieces per row");
        return ROWB >= 256 ? 4 * (t & 3) : 4 * ((t >> 1) & 1);
    }

    __device__ __forceinline__ void setup(const Args &a, int p0, int q0, int wave, int lane)
    {
#pragma unroll
        for (int k = 0; k < DPC; ++k) {
            const int n = k * 4 + wave;                  // DMA instruction index within the chunk
            const int L = n * 64 + lane;                 // 16-byte piece written by this lane
            // Byte offset within the chunk's buffer (its token rows only).  A piece past
            // the last column, or one whose offset would not fit in 32 bits, gets
            // OOR_OFFSET, which no chunk's record count reaches: it reads zero.
            int t, col, ld;
            if (n * 64 < XCH) {
                t = L / (BQ / 8);
                col = q0 + 8 * ((L % (BQ / 8)) ^ swz<XROWB>(t));
                ld = a.d_in;
            } else {
                const int L2 = L - XCH;
                t = L2 / (BP / 8);
                col = p0 + 8 * ((L2 % (BP / 8)) ^ swz<YROWB>(t));
                ld = a.d_out;
            }
            const uint64_t off = ((uint64_t)t * (uint64_t)ld + (uint64_t)col) * 2u;
            voff[k] = (col < ld && off < OOR_OFFSET) ? (uint32_t)off : OOR_OFFSET;
        }
        const int wq = wave % WQ, wp = wave / WQ;
        const int s = lane & 15;
        const int trow = 8 * (lane >> 5) + (s >> 2);     // token row of this lane's 8-byte read
        const int half = (s & 1) * 8;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int qb = wq * 64 + i * 32 + 16 * ((lane >> 4) & 1);
            const int cq = (qb / 8 + ((s & 3) >> 1)) ^ swz<XROWB>(trow);
            ta[i] = trow * XROWB + cq * 16 + half;
            const int pb = wp * 64 + i * 32 + 16 * ((lane >> 4) & 1);
            const int cp = (pb / 8 + ((s & 3) >> 1)) ^ swz<YROWB>(trow);
            tb[i] = XCH * 16 + trow * YROWB + cp * 16 + half;
        }
    }

    // DMA of token chunk c into a stage.  Each chunk gets buffers of its own that start at
    // its first token row and end at its last existing one, so rows past T read zero and
    // no offset grows with the token position.
    __device__ __forceinline__ void issue(const Args &a, unsigned char *stage, int c, int wave)
    {
        const int rows = min(TK, a.T - c * TK);
        const size_t r0 = (size_t)c * TK;
        const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t *>(a.X + r0 * (size_t)a.d_in), (short)0,
            (int)((uint32_t)rows * (uint32_t)a.d_in * 2u), 0x00020000);
        const __amdgpu_buffer_rsrc_t ry = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t *>(a.dY + r0 * (size_t)a.d_out), (short)0,
            (int)((uint32_t)rows * (uint32_t)a.d_out * 2u), 0x00020000);
#pragma unroll
        for (int k = 0; k < DPC; ++k) {
            const int n = k * 4 + wave;
            auto *dst = (__attribute__((address_space(3))) void *)(stage + n * 1024);
            if (n * 64 < XCH)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, dst, 16, voff[k], 0, 0, 0);
            else
                __builtin_amdgcn_raw_ptr_buffer_load_lds(ry, dst, 16, voff[k], 0, 0, 0);
        }
    }

    template <int OFF>
    static __device__ __forceinline__ void tr_read(v4i16_t &r, uint32_t addr)
    {
        asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF) : "memory");
    }

    static __device__ __forceinline__ bf16x8_t cat(v4i16_t lo, v4i16_t hi)
    {
        return __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }

    __device__ __forceinline__ void compute(uint32_t stage_addr)
    {
        v4i16_t fa[2][2][2], fb[2][2][2];                // [k step][sub-tile][token half]
        const uint32_t a0 = stage_addr + ta[0], a1 = stage_addr + ta[1];
        const uint32_t b0 = stage_addr + tb[0], b1 = stage_addr + tb[1];
        tr_read<0 * XROWB>(fa[0][0][0], a0);  tr_read<4 * XROWB>(fa[0][0][1], a0);
        tr_read<0 * XROWB>(fa[0][1][0], a1);  tr_read<4 * XROWB>(fa[0][1][1], a1);
        tr_read<0 * YROWB>(fb[0][0][0], b0);  tr_read<4 * YROWB>(fb[0][0][1], b0);
        tr_read<0 * YROWB>(fb[0][1][0], b1);  tr_read<4 * YROWB>(fb[0][1][1], b1);
        tr_read<16 * XROWB>(fa[1][0][0], a0); tr_read<20 * XROWB>(fa[1][0][1], a0);
        tr_read<16 * XROWB>(fa[1][1][0], a1); tr_read<20 * XROWB>(fa[1][1][1], a1);
        tr_read<16 * YROWB>(fb[1][0][0], b0); tr_read<20 * YROWB>(fb[1][0][1], b0);
        tr_read<16 * YROWB>(fb[1][1][0], b1); tr_read<20 * YROWB>(fb[1][1][1], b1);
        asm volatile("s_waitcnt lgkmcnt(8)"
                     : "+v"(fa[0][0][0]), "+v"(fa[0][0][1]), "+v"(fa[0][1][0]), "+v"(fa[0][1][1]),
                       "+v"(fb[0][0][0]), "+v"(fb[0][0][1]), "+v"(fb[0][1][0]), "+v"(fb[0][1][1]));
#pragma unroll
        for (int iq = 0; iq < 2; ++iq)
#pragma unroll
            for (int ip = 0; ip < 2; ++ip)
                acc[iq][ip] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    cat(fa[0][iq][0], fa[0][iq][1]), cat(fb[0][ip][0], fb[0][ip][1]), acc[iq][ip], 0, 0, 0);
#if FORGE_SCHED_SPLIT
        __builtin_amdgcn_sched_barrier(0);   // keep the first step's MFMAs ahead of the next wait
#endif
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(fa[1][0][0]), "+v"(fa[1][0][1]), "+v"(fa[1][1][0]), "+v"(fa[1][1][1]),
                       "+v"(fb[1][0][0]), "+v"(fb[1][0][1]), "+v"(fb[1][1][0]), "+v"(fb[1][1][1]));
#pragma unroll
        for (int iq = 0; iq < 2; ++iq)
#pragma unroll
            for (int ip = 0; ip < 2; ++ip)
                acc[iq][ip] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    cat(fa[1][iq][0], fa[1][iq][1]), cat(fb[1][ip][0], fb[1][ip][1]), acc[iq][ip], 0, 0, 0);
    }

    // Wait until this wave's DMA for the oldest in-flight chunk has landed (`younger`
    // chunks issued after it may stay in flight), then barrier so every wave's has.
    template <int Y = NS - 2>
    static __device__ __forceinline__ void wait_chunk(int younger)
    {
        static_assert(DPC * (NS - 2) <= 63, "vmcnt range");
        if constexpr (Y == 0) {
            asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
        } else {
            if (younger >= Y) asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"i"(DPC * Y) : "memory");
            else wait_chunk<Y - 1>(younger);
        }
    }

    // Start a tile: zero the accumulators, set up this lane's DMA pieces and fragment
    // offsets, and issue the first NS-1 chunks into the ring.  No barrier.
    __device__ __forceinline__ void begin(const Args &a, int p0, int q0, unsigned char *lds, int wave,
                                          int lane)
    {
#pragma unroll
        for (int iq = 0; iq < 2; ++iq)
#pragma unroll
            for (int ip = 0; ip < 2; ++ip)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[iq][ip][r] = 0.0f;
        const int nch = (a.T + TK - 1) / TK;
        setup(a, p0, q0, wave, lane);
#pragma unroll
        for (int c = 0; c < NS - 1; ++c)
            if (c < nch) issue(a, lds + c * STAGE_BYTES, c, wave);
    }

    // The token loop of a tile started with begin(); executes exactly nch(T) workgroup
    // barriers (one per chunk).
    __device__ __forceinline__ void body(const Args &a, unsigned char *lds, int wave)
    {
        const int nch = (a.T + TK - 1) / TK;
        const uint32_t lds_base = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)lds;
        for (int c = 0; c < nch; ++c) {
            const int younger = min(NS - 2, nch - 1 - c);
            wait_chunk(younger);
#pragma unroll
            for (int h = 0; h < TK / 32; ++h)    // 32 tokens per compute(); X and Y rows of equal length
                compute(lds_base + (uint32_t)((c % NS) * STAGE_BYTES + h * 32 * XROWB));
            if (c + NS - 1 < nch) issue(a, lds + ((c + NS - 1) % NS) * STAGE_BYTES, c + NS - 1, wave);
        }
    }

    // The whole token loop; executes exactly nbar(T, lead) workgroup barriers.  With lead,
    // the first follows the DMA of the first NS-1 chunks: a workgroup's other waves issue
    // their own global loads (the tile's state) after it, so these chunks are queued ahead
    // of them in the CU's vector memory path.  Without state to load (the store-G
    // epilogue) it only delays the mainloop: 1.5 % on the 4096 x 4096 store-G GEMM at
    // T = 4096.
    __device__ __forceinline__ void run(const Args &a, int p0, int q0, unsigned char *lds, int wave,
                                        int lane, bool lead)
    {
        begin(a, p0, q0, lds, wave, lane);
        if (lead) lds_barrier();
        body(a, lds, wave);
        lds_barrier();   // every wave is done reading the stages, which G reuses
    }

    static __device__ __forceinline__ int nch(int T) { return (T + TK - 1) / TK; }
    static __device__ __forceinline__ int nbar(int T, bool lead) { return (T + TK - 1) / TK + (lead ? 2 : 1); }

    // Accumulators -> LDS as G[p][q] (fp32, row pitch GP floats).
    template <int GP>
    __device__ __forceinline__ void stage_g(float *Gs, int wave, int lane) const
    {
        const int wq = wave % WQ, wp = wave / WQ;
#pragma unroll
        for (int iq = 0; iq < 2; ++iq)
#pragma unroll
            for (int ip = 0; ip < 2; ++ip) {
                const int p = wp * 64 + ip * 32 + (lane & 31);
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int q = wq * 64 + iq * 32 + g * 8 + (lane >> 5) * 4;
                    f32x4_t v = {acc[iq][ip][4 * g], acc[iq][ip][4 * g + 1],
                                 acc[iq][ip][4 * g + 2], acc[iq][ip][4 * g + 3]};
                    *reinterpret_cast<f32x4_t *>(Gs + p * GP + q) = v;
                }
            }
    }
};

// ------------------------------------------------------------------------ epilogues

// Lane mapping shared by every epilogue: 256 lanes, each owning 8 consecutive columns of
// one row per pass; consecutive lanes walk a row, so every access is a coalesced 16-byte
// (or 8-byte, int8 codes) vector.
template <int BP, int BQ, int NTH = NROLE>
struct EpiMap {
    static constexpr int GP = BQ + 4;           // LDS G row pitch in floats
    static constexpr int LPR = BQ / 8;          // lanes per row
    static constexpr int RPP = NTH / LPR;       // rows per pass
    static constexpr int NPASS = BP / RPP;
    static constexpr int GS_BYTES = BP * GP * 4;
};

// Per-element update rules of the fused step (the optimizer-family table of App. I; App. D
// measures them by state count).  Each maps (g, w, s1, s2) to (w', s1', s2') in fp32 using
// the scalars of Hyper; NS is the number of state tensors it reads and writes, and W_RW is
// false for the rule that leaves the weight alone (Muon's momentum accumulate: the weight
// update, a Newton--Schulz iteration over the whole buffer, reads state only and runs
// elsewhere).  Decay: AdamW and Lion decay the weight directly (1 - lr wd); the others add
// wd * w to the gradient first, as the common reference implementations do.
template <int E> struct Rule;

template <> struct Rule<EPI_ADAMW> {
    static constexpr int NS = 2;
    static constexpr bool W_RW = true;
    static __device__ __forceinline__ void elem(float g, float w, float s1, float s2, const Hyper &h,
                                                float &w1, float &t1, float &t2)
    {
        float rv;
        adamw_elem(g, w, s1, s2, h, w1, t1, t2, rv);
    }
};

template <> struct Rule<EPI_SGD> {            // w' = w - lr (g + wd w)
    static constexpr int NS = 0;
    static constexpr bool W_RW = true;
    static __device__ __forceinline__ void elem(float g, float w, float, float, const Hyper &h,
                                                float &w1, float &, float &)
    {
        const float gg = __builtin_fmaf(h.wd, w, g);
        w1 = __builtin_fmaf(-h.lr, gg, w);
    }
};

template <> struct Rule<EPI_SGDM> {           // b' = mu b + (g + wd w); w' = w - lr b'
    static constexpr int NS = 1;
    static constexpr bool W_RW = true;
    static __device__ __forceinline__ void elem(float g, float w, float s1, float, const Hyper &h,
                                                float &w1, float &t1, float &)
    {
        const float gg = __builtin_fmaf(h.wd, w, g);
        t1 = __builtin_fmaf(h.b1, s1, gg);
        w1 = __builtin_fmaf(-h.lr, t1, w);
    }
};

template <> struct Rule<EPI_ADAGRAD> {        // s' = s + gg^2; w' = w - clr gg / (sqrt(s') + eps)
    static constexpr int NS = 1;
    static constexpr bool W_RW = true;
    static __device__ __forceinline__ void elem(float g, float w, float s1, float, const Hyper &h,
                                                float &w1, float &t1, float &)
    {
        const float gg = __builtin_fmaf(h.wd, w, g);
        t1 = __builtin_fmaf(gg, gg, s1);
        const float den = __builtin_amdgcn_sqrtf(t1) + h.eps;
        w1 = __builtin_fmaf(-(h.lr * gg), __builtin_amdgcn_rcpf(den), w);
    }
};

template <> struct Rule<EPI_RMSPROP> {        // v' = a v + (1-a) gg^2; w' = w - lr gg / (sqrt(v') + eps)
    static constexpr int NS = 1;
    static constexpr bool W_RW = true;
    static __device__ __forceinline__ void elem(float g, float w, float s1, float, const Hyper &h,
                                                float &w1, float &t1, float &)
    {
        const float gg = __builtin_fmaf(h.wd, w, g);
        t1 = __builtin_fmaf(h.b2, s1, (h.c2 * gg) * gg);
        const float den = __builtin_amdgcn_sqrtf(t1) + h.eps;
        w1 = __builtin_fmaf(-(h.lr * gg), __builtin_amdgcn_rcpf(den), w);
    }
};

template <> struct Rule<EPI_LION> {           // w' = (1 - lr wd) w - lr sign(b1 m + (1-b1) g); m' = b2 m + (1-b2) g
    static constexpr int NS = 1;
    static constexpr bool W_RW = true;
    static __device__ __forceinline__ void elem(float g, float w, float s1, float, const Hyper &h,
                                                float &w1, float &t1, float &)
    {
        const float c = __builtin_fmaf(h.b1, s1, h.c1 * g);
        const float sg = c > 0.0f ? 1.0f : (c < 0.0f ? -1.0f : c);   // sign; 0 and NaN pass through
        w1 = __builtin_fmaf(h.wdf, w, -(h.lr * sg));
        t1 = __builtin_fmaf(h.b2, s1, h.c2 * g);
    }
};

template <> struct Rule<EPI_NADAM> {          // Adam moments of gg; w' = w - (ka gg + kb m') / (sqrt(v'/bc2) + eps)
    static constexpr int NS = 2;
    static constexpr bool W_RW = true;
    static __device__ __forceinline__ void elem(float g, float w, float s1, float s2, const Hyper &h,
                                                float &w1, float &t1, float &t2)
    {
        const float gg = __builtin_fmaf(h.wd, w, g);
        t1 = __builtin_fmaf(h.b1, s1, h.c1 * gg);
        t2 = __builtin_fmaf(h.b2, s2, (h.c2 * gg) * gg);
        const float den = __builtin_fmaf(__builtin_amdgcn_sqrtf(t2), h.inv_sqrt_bc2, h.eps);
        const float num = __builtin_fmaf(h.ka, gg, h.kb * t1);
        w1 = __builtin_fmaf(-num, __builtin_amdgcn_rcpf(den), w);
    }
};

template <> struct Rule<EPI_RADAM> {          // Adam moments of gg; w' = w - ka m' / (sqrt(v') + eps) - kb m'
    static constexpr int NS = 2;
    static constexpr bool W_RW = true;
    static __device__ __forceinline__ void elem(float g, float w, float s1, float s2, const Hyper &h,
                                                float &w1, float &t1, float &t2)
    {
        const float gg = __builtin_fmaf(h.wd, w, g);
        t1 = __builtin_fmaf(h.b1, s1, h.c1 * gg);
        t2 = __builtin_fmaf(h.b2, s2, (h.c2 * gg) * gg);
        const float den = __builtin_amdgcn_sqrtf(t2) + h.eps;
        const float upd = __builtin_fmaf(h.ka * t1, __builtin_amdgcn_rcpf(den), h.kb * t1);
        w1 = w - upd;
    }
};

template <> struct Rule<EPI_ADAMAX> {         // m' = b1 m + (1-b1) gg; u' = max(b2 u, |gg| + eps); w' = w - lr/bc1 m'/u'
    static constexpr int NS = 2;
    static constexpr bool W_RW = true;
    static __device__ __forceinline__ void elem(float g, float w, float s1, float s2, const Hyper &h,
                                                float &w1, float &t1, float &t2)
    {
        const float gg = __builtin_fmaf(h.wd, w, g);
        t1 = __builtin_fmaf(h.b1, s1, h.c1 * gg);
        t2 = __builtin_fmaxf(h.b2 * s2, __builtin_fabsf(gg) + h.eps);
        w1 = __builtin_fmaf(-(h.lr_bc1 * t1), __builtin_amdgcn_rcpf(t2), w);
    }
};

template <> struct Rule<EPI_MUON> {           // B' = mu B + G (the GEMM's beta); W untouched
    static constexpr int NS = 1;
    static constexpr bool W_RW = false;
    static __device__ __forceinline__ void elem(float g, float, float s1, float, const Hyper &h,
                                                float &, float &t1, float &)
    {
        t1 = __builtin_fmaf(h.b1, s1, g);
    }
};

// The epilogue of a rule on fp32 or bf16 state.  The stream waves prefetch the tile's
// W and state into registers while the mainloop runs (bf16 state: six or eight of the
// eight row passes; fp32 state, twice the bytes: four), then each lane updates 8
// consecutive columns of one row per pass, loading later passes' state a fixed number of
// passes ahead.
// Byte offset of element (p, q) of a [rows, ld] tensor with `eb`-byte elements, or an
// offset past every buffer end (reads zero) when the element lies outside the tensor.
__device__ __forceinline__ uint32_t elem_off(int p, int q, int rows, int ld, int eb)
{
    if (p >= rows || q >= ld) return OOR_OFFSET;
    const uint64_t off = ((uint64_t)p * (uint64_t)ld + (uint64_t)q) * (uint64_t)eb;
    return off < OOR_OFFSET ? (uint32_t)off : OOR_OFFSET;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_of(const void *base, uint64_t bytes)
{
    const uint32_t n = bytes < OOR_OFFSET ? (uint32_t)bytes : OOR_OFFSET;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)n, 0x00020000);
}

template <int BP, int BQ, int MK, int E, int AH = 0>
struct EpiRule {
    using M = EpiMap<BP, BQ>;
    using R = Rule<E>;
    static_assert(MK == MK_BF16 || MK == MK_F32, "the rule epilogue keeps bf16 or fp32 state");
    static constexpr bool F32 = (MK == MK_F32);
    static constexpr int NPF = M::NPASS;
    // Row passes whose state is loaded while the mainloop runs (bf16 state: AH, or by
    // default all but two); the loads of the others are issued as the epilogue starts,
    // AHEAD passes before their use.  Less state in flight per CU suits in-place HBM
    // traffic, fewer than six passes loses overlap with the GEMM; the launcher picks all
    // eight for long launches.  fp32 state: four passes, 80 B per lane each with the bf16 W
    // (at most 128 VGPRs; on the 4096 x 4096 microbenchmark AdamW took 99.5-99.8 against
    // 106 us at T = 512 and SGD with momentum 58.7-58.9 against 65.5 us, with no prefetch).
#ifdef FORGE_PF_AHEAD
    static constexpr int AHEAD = FORGE_PF_AHEAD < M::NPASS ? FORGE_PF_AHEAD : M::NPASS;
#else
    static constexpr int AHEAD = F32 ? 4
                               : AH > 0 ? (AH < M::NPASS ? AH : M::NPASS) : (M::NPASS > 2 ? M::NPASS - 2 : M::NPASS);
#endif
    // packed bf16 state: one 16-byte word per pass and lane; fp32 state: two
    static constexpr int SW = F32 ? 2 : 1;
    u32x4_t pw[R::W_RW ? NPF : 1], ps1[R::NS >= 1 ? NPF : 1][SW], ps2[R::NS >= 2 ? NPF : 1][SW];

    // Loads of pass I (one row per lane) into the prefetch registers.
    template <int I>
    __device__ __forceinline__ void prefetch_pass(const Args &a, int p0, int q0, int s)
    {
        // buffer loads: elements outside the matrix read as zero
        const int rs = s / M::LPR, q = q0 + (s % M::LPR) * 8;
        const int p = p0 + I * M::RPP + rs;
        const uint64_t n = 2ull * (uint64_t)a.d_out * (uint64_t)a.d_in;
        const uint32_t off = elem_off(p, q, a.d_out, a.d_in, 2);
        if constexpr (R::W_RW) pw[I] = __builtin_amdgcn_raw_buffer_load_b128(rsrc_of(a.W, n), off, 0, 2);
        if constexpr (!F32) {
            if constexpr (R::NS >= 1) ps1[I][0] = __builtin_amdgcn_raw_buffer_load_b128(rsrc_of(a.m, n), off, 0, 2);
            if constexpr (R::NS >= 2) ps2[I][0] = __builtin_amdgcn_raw_buffer_load_b128(rsrc_of(a.v, n), off, 0, 2);
        } else {
            // an fp32 tensor may pass 4 GB, beyond a buffer's 32-bit offsets: loads
            // masked to the matrix, zero outside it
            const bool ok = p < a.d_out && q < a.d_in;
            const size_t e = (size_t)p * a.d_in + q;
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                if constexpr (R::NS >= 1) ps1[I][k] = u32x4_t{0u, 0u, 0u, 0u};
                if constexpr (R::NS >= 2) ps2[I][k] = u32x4_t{0u, 0u, 0u, 0u};
            }
            if (ok) {
#pragma unroll
                for (int k = 0; k < 2; ++k) {
                    if constexpr (R::NS >= 1) ps1[I][k] = ld_nt<u32x4_t>(static_cast<const float *>(a.m) + e + 4 * k);
                    if constexpr (R::NS >= 2) ps2[I][k] = ld_nt<u32x4_t>(static_cast<const float *>(a.v) + e + 4 * k);
                }
            }
        }
    }

    template <int I = 0>
    __device__ __forceinline__ void prefetch(const Args &a, int p0, int q0, int s)
    {
        prefetch_pass<I>(a, p0, q0, s);
        if constexpr (I + 1 < AHEAD) prefetch<I + 1>(a, p0, q0, s);
    }

    // prefetch_pass<i> for a pass index known once the caller's loop is unrolled.
    template <int I = 0>
    __device__ __forceinline__ void prefetch_at(int i, const Args &a, int p0, int q0, int s)
    {
        if (i == I) prefetch_pass<I>(a, p0, q0, s);
        else if constexpr (I + 1 < M::NPASS) prefetch_at<I + 1>(i, a, p0, q0, s);
    }

    // Element e of 8 consecutive values held as packed bf16 pairs, or as two fp32 quads.
    static __device__ __forceinline__ float elt(const u32x4_t &u, int e)
    {
        return (e & 1) ? bf_hi(u[e >> 1]) : bf_lo(u[e >> 1]);
    }
    static __device__ __forceinline__ float elt(const f32x4_t &x0, const f32x4_t &x1, int e)
    {
        return e < 4 ? x0[e] : x1[e - 4];
    }

    static __device__ __forceinline__ void store_state(void *base, size_t off, const float (&f)[8])
    {
        if constexpr (MK == MK_BF16) {
            u32x4_t u;
#pragma unroll
            for (int k = 0; k < 4; ++k) u[k] = pack_bf16(f[2 * k], f[2 * k + 1]);
            st_nt<u32x4_t>(static_cast<uint16_t *>(base) + off, u);
        } else {
            float *p = static_cast<float *>(base) + off;
            st_nt<f32x4_t>(p, f32x4_t{f[0], f[1], f[2], f[3]});
            st_nt<f32x4_t>(p + 4, f32x4_t{f[4], f[5], f[6], f[7]});
        }
    }

    __device__ __forceinline__ void run(const Args &a, int p0, int q0, int s, const float *Gs)
    {
        const int rs = s / M::LPR, qo = (s % M::LPR) * 8, q = q0 + qo;
        const Hyper h = a.h;
#pragma unroll
        for (int i = 0; i < M::NPASS; ++i) {
            if (i + AHEAD < M::NPASS) prefetch_at(i + AHEAD, a, p0, q0, s);
            const int p = p0 + i * M::RPP + rs;
            const bool ok = q < a.d_in && p < a.d_out;
            const size_t off = (size_t)p * a.d_in + q;
            const float *gr = Gs + (i * M::RPP + rs) * M::GP + qo;
            const f32x4_t g0 = *reinterpret_cast<const f32x4_t *>(gr);
            const f32x4_t g1 = *reinterpret_cast<const f32x4_t *>(gr + 4);
            // W and the states stay packed until each element is needed
            u32x4_t w4 = {0u, 0u, 0u, 0u}, a4 = w4, b4 = w4;
            f32x4_t a0 = {0, 0, 0, 0}, a1 = a0, b0 = a0, b1 = a0;
            if constexpr (F32) {
                if constexpr (R::W_RW) w4 = pw[i];
                if constexpr (R::NS >= 1) {
                    a0 = __builtin_bit_cast(f32x4_t, ps1[i][0]);
                    a1 = __builtin_bit_cast(f32x4_t, ps1[i][1]);
                }
                if constexpr (R::NS >= 2) {
                    b0 = __builtin_bit_cast(f32x4_t, ps2[i][0]);
                    b1 = __builtin_bit_cast(f32x4_t, ps2[i][1]);
                }
            } else {
                if constexpr (R::W_RW) w4 = pw[i];
                if constexpr (R::NS >= 1) a4 = ps1[i][0];
                if constexpr (R::NS >= 2) b4 = ps2[i][0];
            }
            float wo[8], o1[8], o2[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float g = elt(g0, g1, e);
                const float w = R::W_RW ? elt(w4, e) : 0.0f;
                const float x = R::NS >= 1 ? (F32 ? elt(a0, a1, e) : elt(a4, e)) : 0.0f;
                const float y = R::NS >= 2 ? (F32 ? elt(b0, b1, e) : elt(b4, e)) : 0.0f;
                R::elem(g, w, x, y, h, wo[e], o1[e], o2[e]);
            }
            if (ok) {
                if constexpr (R::W_RW) {
                    u32x4_t wn;
#pragma unroll
                    for (int k = 0; k < 4; ++k) wn[k] = pack_bf16(wo[2 * k], wo[2 * k + 1]);
                    st_nt<u32x4_t>(a.W + off, wn);
                }
                if constexpr (R::NS >= 1) store_state(a.m, off, o1);
                if constexpr (R::NS >= 2) store_state(a.v, off, o2);
            }
        }
    }
};

template <int BP, int BQ, int MK>
using EpiAdamW = EpiRule<BP, BQ, MK, EPI_ADAMW>;

// The absmax reductions below run on the bit patterns of non-negative floats (+0 and up),
// whose signed-integer order is their numeric order.
//
// Lane exchange within a row of 16 lanes (DPP; no LDS round trip).  CTRL is a DPP control:
// 0xB1 and 0x4E are the quad permutations [1,0,3,2] and [2,3,0,1], 0x141 mirrors each half
// row of 8 lanes, 0x128 rotates the row by 8.
template <int CTRL>
__device__ __forceinline__ int dpp_i(int x)
{
    return __builtin_amdgcn_mov_dpp(x, CTRL, 0xF, 0xF, true);
}

// Max of x >= 0 over each aligned group of 8 lanes, returned to all 8 (every lane active).
__device__ __forceinline__ float max8(float x)
{
    int b = __float_as_int(x);
    b = max(b, dpp_i<0xB1>(b));
    b = max(b, dpp_i<0x4E>(b));
    return __int_as_float(max(b, dpp_i<0x141>(b)));
}

// int8 codes of eight values y = x / s: clamped to [lo, 127] (lo = -127 for m; for sqrt(v)
// or v, 1 in a non-zero block and 0 in an all-zero one), rounded to nearest even, packed.
// Clamping before rounding gives the same integer, as both bounds are integers.  Adding
// 1.5 * 2^23 does the rounding (the sum's ulp is 1) and leaves the integer's two's-
// complement low byte as the sum's low byte.
__device__ __forceinline__ u32x2_t pack_codes(const float (&y)[8], const float (&lo)[8])
{
    uint32_t b[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) b[e] = __float_as_uint(__builtin_amdgcn_fmed3f(y[e], lo[e], 127.0f) + 12582912.0f);
    u32x2_t r;
#pragma unroll
    for (int k = 0; k < 2; ++k)
        r[k] = __builtin_amdgcn_perm(b[4 * k + 1], b[4 * k], 0x0c0c0400u) |
               __builtin_amdgcn_perm(b[4 * k + 3], b[4 * k + 2], 0x04000c0cu);
    return r;
}
__device__ __forceinline__ u32x2_t pack_codes(const float (&y)[8], float lo)
{
    const float l[8] = {lo, lo, lo, lo, lo, lo, lo, lo};
    return pack_codes(y, l);
}

// x / 127 in fp32, correctly rounded for every finite x >= 0: the product with RN(1/127)
// and one fma correction from its exact remainder.  Checked against IEEE division over
// every non-negative finite float.
__device__ __forceinline__ float div127(float x)
{
    constexpr float R = 1.0f / 127.0f;
    const float q = x * R;
    return __builtin_fmaf(__builtin_fmaf(-q, 127.0f, x), R, q);
}

// AdamW on int8 moments in the 64-wide row-block layout of App. B: one fp32 scale per 64
// consecutive elements of a row, m = s_m q_m and v = s_v q_v (v stored itself).  A block is
// exactly the 8 consecutive lanes that hold its row's 64 columns in one pass, so the new
// block absmax closes with three DPP exchanges and each row is dequantised, updated and
// re-quantised in a single pass: s = absmax / 127 (fp32, correctly rounded),
// q = round_half_even(x * RN(1/s)) (the fp32 reciprocal of the scale, not a division)
// clamped to [-127, 127], v codes at least 1 in a non-zero block.
// The weight update reads the unquantised fp32 m', v'.
template <int BP, int BQ>
struct EpiI8Row {
    using M = EpiMap<BP, BQ>;
    static_assert(BQ % I8_ROW_BLOCK == 0 && M::LPR * 8 == BQ, "a block is 8 lanes of one row");
    u32x4_t pw[M::NPASS];
    u32x2_t pm[M::NPASS], pv[M::NPASS];
    float sm[M::NPASS], sv[M::NPASS];

    static __device__ __forceinline__ int nblocks(const Args &a) { return (a.d_in + I8_ROW_BLOCK - 1) / I8_ROW_BLOCK; }

    template <int I>
    __device__ __forceinline__ void prefetch_pass(const Args &a, int p0, int q0, int s)
    {
        // buffer loads: elements outside the matrix read as zero
        const int rs = s / M::LPR, q = q0 + (s % M::LPR) * 8;
        const int p = p0 + I * M::RPP + rs, nb = nblocks(a);
        const uint64_t n = (uint64_t)a.d_out * (uint64_t)a.d_in, ns = 4ull * (uint64_t)a.d_out * (uint64_t)nb;
        const uint32_t off = elem_off(p, q, a.d_out, a.d_in, 1);
        const uint32_t so = q < a.d_in ? elem_off(p, q / I8_ROW_BLOCK, a.d_out, nb, 4) : OOR_OFFSET;
        pw[I] = __builtin_amdgcn_raw_buffer_load_b128(rsrc_of(a.W, 2ull * n), off == OOR_OFFSET ? off : 2u * off, 0, 2);
        pm[I] = __builtin_amdgcn_raw_buffer_load_b64(rsrc_of(a.m, n), off, 0, 2);
        pv[I] = __builtin_amdgcn_raw_buffer_load_b64(rsrc_of(a.v, n), off, 0, 2);
        sm[I] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc_of(a.ms, ns), so, 0, 0));
        sv[I] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc_of(a.vs, ns), so, 0, 0));
    }

    template <int I = 0>
    __device__ __forceinline__ void prefetch(const Args &a, int p0, int q0, int s)
    {
        prefetch_pass<I>(a, p0, q0, s);
        if constexpr (I + 1 < M::NPASS) prefetch<I + 1>(a, p0, q0, s);
    }

    static __device__ __forceinline__ float code_at(u32x2_t c, int e)
    {
        return (float)(int8_t)((c[e >> 2] >> (8 * (e & 3))) & 0xFFu);
    }

    __device__ __forceinline__ void run(const Args &a, int p0, int q0, int s, const float *Gs)
    {
        const int rs = s / M::LPR, qo = (s % M::LPR) * 8, q = q0 + qo;
        const Hyper h = a.h;
#pragma unroll
        for (int i = 0; i < M::NPASS; ++i) {
            const int p = p0 + i * M::RPP + rs;
            const bool ok = q < a.d_in && p < a.d_out;
            const float *gr = Gs + (i * M::RPP + rs) * M::GP + qo;
            const f32x4_t g0 = *reinterpret_cast<const f32x4_t *>(gr);
            const f32x4_t g1 = *reinterpret_cast<const f32x4_t *>(gr + 4);
            float wo[8], mo[8], vo[8];
            float am = 0.0f, av = 0.0f;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float g = e < 4 ? g0[e] : g1[e - 4];
                const float w = (e & 1) ? bf_hi(pw[i][e >> 1]) : bf_lo(pw[i][e >> 1]);
                float rv;
                adamw_elem(g, w, sm[i] * code_at(pm[i], e), sv[i] * code_at(pv[i], e), h, wo[e], mo[e], vo[e], rv);
                am = fmaxf(am, fabsf(mo[e]));
                av = fmaxf(av, vo[e]);
            }
            if (!ok) am = av = 0.0f;
            am = max8(am);
            av = max8(av);
            const float scm = div127(am), scv = div127(av);
            const float rcm = scm > 0.0f ? __builtin_amdgcn_rcpf(scm) : 0.0f;
            const float rcv = scv > 0.0f ? __builtin_amdgcn_rcpf(scv) : 0.0f;
            float ym[8], yv[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                ym[e] = mo[e] * rcm;
                yv[e] = vo[e] * rcv;
            }
            const u32x2_t cm = pack_codes(ym, -127.0f), cv = pack_codes(yv, rcv > 0.0f ? 1.0f : 0.0f);
            if (ok) {
                const size_t off = (size_t)p * a.d_in + q;
                u32x4_t wn;
#pragma unroll
                for (int k = 0; k < 4; ++k) wn[k] = pack_bf16(wo[2 * k], wo[2 * k + 1]);
                st_nt<u32x4_t>(a.W + off, wn);
                st_nt<u32x2_t>(static_cast<int8_t *>(a.m) + off, cm);
                st_nt<u32x2_t>(static_cast<int8_t *>(a.v) + off, cv);
                if ((s & 7) == 0) {
                    const size_t so = (size_t)p * nblocks(a) + q / I8_ROW_BLOCK;
                    a.ms[so] = scm;
                    a.vs[so] = scv;
                }
            }
        }
    }
};

// fp8 tensors: OCP E4M3 codes (largest finite 448, round to nearest even; the hardware
// conversion gives NaN past 464, so values are clamped into range first) with one scale per
// tensor, s = amax / 448, where amax is a previous step's max |x| over the tensor (delayed
// scaling; a scale of 1 while there is no history).  Each tensor has a ring of four amax
// slots: step t decodes with the scale of slot (t-2)%4 (the one its stored codes were written
// with), encodes with slot (t-1)%4, max-reduces its own new values into slot t%4 and clears
// slot (t+1)%4 for the next step, so that no slot is read while another workgroup writes it.
struct Fp8 {
    static __device__ __forceinline__ float scale_of(float amax) { return amax > 0.0f ? amax / 448.0f : 1.0f; }
    static __device__ __forceinline__ float clamp(float x) { return fminf(fmaxf(x, -448.0f), 448.0f); }
    // value of byte e of 8 packed codes
    static __device__ __forceinline__ float decode(const u32x2_t &c, int e)
    {
        const int w = (int)c[e >> 2];
        switch (e & 3) {
        case 0: return __builtin_amdgcn_cvt_f32_fp8(w, 0);
        case 1: return __builtin_amdgcn_cvt_f32_fp8(w, 1);
        case 2: return __builtin_amdgcn_cvt_f32_fp8(w, 2);
        default: return __builtin_amdgcn_cvt_f32_fp8(w, 3);
        }
    }
    // 8 values (already scaled) -> 8 codes
    static __device__ __forceinline__ u32x2_t encode8(const float (&x)[8])
    {
        u32x2_t c;
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(clamp(x[4 * k]), clamp(x[4 * k + 1]), 0, false);
            c[k] = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(clamp(x[4 * k + 2]), clamp(x[4 * k + 3]), lo, true);
        }
        return c;
    }
    // Record a wave's amax into the slot (one atomic per wave, skipped when the slot already
    // holds at least as much; amax >= 0, so its bit pattern orders like the value).
    static __device__ __forceinline__ void record(float *ring, int slot, float amax, int lane)
    {
#pragma unroll
        for (int d = 32; d > 0; d >>= 1) amax = fmaxf(amax, __shfl_xor(amax, d));
        if (lane == 0) {
            unsigned *p = reinterpret_cast<unsigned *>(ring + slot);
            const unsigned bits = __float_as_uint(amax);
            if (bits > __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) atomicMax(p, bits);
        }
    }
};

// AdamW with fp8 weights (WF8) and / or fp8 moments (MF8; m and sqrt(v) stored, the sqrt(v)
// codes at least the smallest positive code when v' > 0); the other tensors bf16.  The
// update reads the decoded state and runs in fp32 as everywhere else.
template <int BP, int BQ, bool WF8, bool MF8>
struct EpiQ {
    using M = EpiMap<BP, BQ>;
    static constexpr int N16W = WF8 ? 1 : M::NPASS, N8W = WF8 ? M::NPASS : 1;
    static constexpr int N16M = MF8 ? 1 : M::NPASS, N8M = MF8 ? M::NPASS : 1;
    u32x4_t pw16[N16W], pm16[N16M], pv16[N16M];
    u32x2_t pw8[N8W], pm8[N8M], pv8[N8M];
    bool first_tile = false;       // the matrix's first tile clears the next step's slots

    template <int I>
    __device__ __forceinline__ void prefetch_pass(const Args &a, int p0, int q0, int s)
    {
        const int rs = s / M::LPR, q = q0 + (s % M::LPR) * 8;
        const int p = p0 + I * M::RPP + rs;
        const u32x4_t z4 = {0u, 0u, 0u, 0u};
        const u32x2_t z2 = {0u, 0u};
        if constexpr (WF8) pw8[I] = z2; else pw16[I] = z4;
        if constexpr (MF8) { pm8[I] = z2; pv8[I] = z2; } else { pm16[I] = z4; pv16[I] = z4; }
        if (q < a.d_in && p < a.d_out) {
            const size_t off = (size_t)p * a.d_in + q;
            if constexpr (WF8) pw8[I] = ld_nt<u32x2_t>(reinterpret_cast<const uint8_t *>(a.W) + off);
            else pw16[I] = ld_nt<u32x4_t>(a.W + off);
            if constexpr (MF8) {
                pm8[I] = ld_nt<u32x2_t>(static_cast<const uint8_t *>(a.m) + off);
                pv8[I] = ld_nt<u32x2_t>(static_cast<const uint8_t *>(a.v) + off);
            } else {
                pm16[I] = ld_nt<u32x4_t>(static_cast<const uint16_t *>(a.m) + off);
                pv16[I] = ld_nt<u32x4_t>(static_cast<const uint16_t *>(a.v) + off);
            }
        }
    }

    template <int I = 0>
    __device__ __forceinline__ void prefetch(const Args &a, int p0, int q0, int s)
    {
        prefetch_pass<I>(a, p0, q0, s);
        if constexpr (I + 1 < M::NPASS) prefetch<I + 1>(a, p0, q0, s);
    }

    static __device__ __forceinline__ float bf(const u32x4_t &u, int e)
    {
        return (e & 1) ? bf_hi(u[e >> 1]) : bf_lo(u[e >> 1]);
    }

    __device__ __forceinline__ void run(const Args &a, int p0, int q0, int s, const float *Gs)
    {
        const int rs = s / M::LPR, qo = (s % M::LPR) * 8, q = q0 + qo;
        const Hyper h = a.h;
        const int wslot = a.slot, enc = (a.slot + 3) % AMAX_SLOTS, dec = (a.slot + 2) % AMAX_SLOTS;
        float w_dec = 1.0f, w_inv = 1.0f, m_dec = 1.0f, m_inv = 1.0f, v_dec = 1.0f, v_inv = 1.0f;
        if constexpr (WF8) {
            w_dec = Fp8::scale_of(a.wr[dec]);
            w_inv = 1.0f / Fp8::scale_of(a.wr[enc]);
        }
        if constexpr (MF8) {
            m_dec = Fp8::scale_of(a.ms[dec]);
            m_inv = 1.0f / Fp8::scale_of(a.ms[enc]);
            v_dec = Fp8::scale_of(a.vs[dec]);
            v_inv = 1.0f / Fp8::scale_of(a.vs[enc]);
        }
        float aw = 0.0f, am = 0.0f, av = 0.0f;
#pragma unroll
        for (int i = 0; i < M::NPASS; ++i) {
            const int p = p0 + i * M::RPP + rs;
            const bool ok = q < a.d_in && p < a.d_out;
            const float *gr = Gs + (i * M::RPP + rs) * M::GP + qo;
            const f32x4_t g0 = *reinterpret_cast<const f32x4_t *>(gr);
            const f32x4_t g1 = *reinterpret_cast<const f32x4_t *>(gr + 4);
            float wo[8], mo[8], vo[8], ro[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float g = e < 4 ? g0[e] : g1[e - 4];
                const float w = WF8 ? w_dec * Fp8::decode(pw8[i], e) : bf(pw16[i], e);
                float m0, v0;
                if constexpr (MF8) {
                    m0 = m_dec * Fp8::decode(pm8[i], e);
                    const float r0 = v_dec * Fp8::decode(pv8[i], e);
                    v0 = r0 * r0;
                } else {
                    m0 = bf(pm16[i], e);
                    v0 = bf(pv16[i], e);
                }
                adamw_elem(g, w, m0, v0, h, wo[e], mo[e], vo[e], ro[e]);
            }
            if (ok) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    aw = fmaxf(aw, fabsf(wo[e]));
                    am = fmaxf(am, fabsf(mo[e]));
                    av = fmaxf(av, ro[e]);
                }
                const size_t off = (size_t)p * a.d_in + q;
                if constexpr (WF8) {
                    float x[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) x[e] = wo[e] * w_inv;
                    st_nt<u32x2_t>(reinterpret_cast<uint8_t *>(a.W) + off, Fp8::encode8(x));
                } else {
                    u32x4_t wn;
#pragma unroll
                    for (int k = 0; k < 4; ++k) wn[k] = pack_bf16(wo[2 * k], wo[2 * k + 1]);
                    st_nt<u32x4_t>(a.W + off, wn);
                }
                if constexpr (MF8) {
                    float xm[8], xv[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        xm[e] = mo[e] * m_inv;
                        xv[e] = ro[e] * v_inv;
                    }
                    u32x2_t cv = Fp8::encode8(xv);
#pragma unroll
                    for (int e = 0; e < 8; ++e)      // sqrt(v') > 0 never stores as zero
                        if (ro[e] > 0.0f && ((cv[e >> 2] >> (8 * (e & 3))) & 0x7Fu) == 0u)
                            cv[e >> 2] |= 1u << (8 * (e & 3));
                    st_nt<u32x2_t>(static_cast<uint8_t *>(a.m) + off, Fp8::encode8(xm));
                    st_nt<u32x2_t>(static_cast<uint8_t *>(a.v) + off, cv);
                } else {
                    u32x4_t mn, vn;
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        mn[k] = pack_bf16(mo[2 * k], mo[2 * k + 1]);
                        vn[k] = pack_bf16(vo[2 * k], vo[2 * k + 1]);
                    }
                    st_nt<u32x4_t>(static_cast<uint16_t *>(a.m) + off, mn);
                    st_nt<u32x4_t>(static_cast<uint16_t *>(a.v) + off, vn);
                }
            }
        }
        const int lane = s & 63;
        if constexpr (WF8) Fp8::record(a.wr, wslot, aw, lane);
        if constexpr (MF8) {
            Fp8::record(a.ms, wslot, am, lane);
            Fp8::record(a.vs, wslot, av, lane);
        }
        if (first_tile && s == 0) {
            const int clr = (a.slot + 1) % AMAX_SLOTS;
            if constexpr (WF8) a.wr[clr] = 0.0f;
            if constexpr (MF8) {
                a.ms[clr] = 0.0f;
                a.vs[clr] = 0.0f;
            }
        }
    }
};

template <class T> struct IsEpiQ { static constexpr bool value = false; };
template <int BP, int BQ, bool W, bool M> struct IsEpiQ<EpiQ<BP, BQ, W, M>> { static constexpr bool value = true; };

// The epilogue of (moment kind, rule): the row-block int8 layout and the fp8 encodings have
// their own (AdamW only).
template <int BP, int BQ, int MK, int E, int AH = 0> struct EpiSel { using T = EpiRule<BP, BQ, MK, E, AH>; };
template <int BP, int BQ> struct EpiSel<BP, BQ, MK_I8R64, EPI_ADAMW> { using T = EpiI8Row<BP, BQ>; };
template <int BP, int BQ> struct EpiSel<BP, BQ, MK_FP8, EPI_ADAMW> { using T = EpiQ<BP, BQ, false, true>; };
template <int BP, int BQ> struct EpiSel<BP, BQ, MK_BF16, EPI_ADAMW_WFP8> { using T = EpiQ<BP, BQ, true, false>; };
template <int BP, int BQ> struct EpiSel<BP, BQ, MK_FP8, EPI_ADAMW_WFP8> { using T = EpiQ<BP, BQ, true, true>; };

// AdamW on int8 block-absmax moments (App. B scheme; blocks of 256 rows along d_out,
// second moment stored through its square root, codes of v floored at 1).  The tile is
// one block tall, so each column's absmax is a reduction over the tile's 256 rows:
// lanes of a wave first (shuffles), then the four stream waves (LDS).  Pass 1 updates W
// and collects the absmax; pass 2 recomputes the same fp32 m', sqrt(v') and quantises.
template <int BP, int BQ>
struct EpiAdamWI8 {
    using M = EpiMap<BP, BQ>;
    static_assert(BP == I8_BLOCK, "an int8 tile is one scale block tall");
    static constexpr int RED_BYTES = 2 * 4 * BQ * 4;     // [m|v][stream wave][column]
    u32x4_t pw[M::NPASS];
    u32x2_t pm[M::NPASS], pv[M::NPASS];
    float sm[8], sv[8];

    // Loads are range-checked buffer loads: elements outside the matrix read as zero, and no
    // branch splits the code per row.
    __device__ __forceinline__ void load_w(const Args &a, int p0, int q0, int s, int i)
    {
        const int p = p0 + i * M::RPP + s / M::LPR, q = q0 + (s % M::LPR) * 8;
        const uint64_t n = 2ull * (uint64_t)a.d_out * (uint64_t)a.d_in;
        pw[i] = __builtin_amdgcn_raw_buffer_load_b128(rsrc_of(a.W, n), elem_off(p, q, a.d_out, a.d_in, 2), 0, 2);
    }

    __device__ __forceinline__ void prefetch(const Args &a, int p0, int q0, int s)
    {
        const int rs = s / M::LPR, q = q0 + (s % M::LPR) * 8;
        const uint64_t n = (uint64_t)a.d_out * (uint64_t)a.d_in;
#pragma unroll
        for (int i = 0; i < M::NPASS; ++i) {
            const int p = p0 + i * M::RPP + rs;
            load_w(a, p0, q0, s, i);
            const uint32_t off = elem_off(p, q, a.d_out, a.d_in, 1);
            pm[i] = __builtin_amdgcn_raw_buffer_load_b64(rsrc_of(a.m, n), off, 0, 2);
            pv[i] = __builtin_amdgcn_raw_buffer_load_b64(rsrc_of(a.v, n), off, 0, 2);
        }
        const int blk = p0 / I8_BLOCK, nblk = (a.d_out + I8_BLOCK - 1) / I8_BLOCK;
        const uint64_t ns = 4ull * (uint64_t)nblk * (uint64_t)a.d_in;
        const uint32_t so = elem_off(blk, q, nblk, a.d_in, 4);
        const __amdgpu_buffer_rsrc_t rm = rsrc_of(a.ms, ns), rv = rsrc_of(a.vs, ns);
        const uint32_t so4 = so == OOR_OFFSET ? so : so + 16u;
        const f32x4_t s0 = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rm, so, 0, 2));
        const f32x4_t s1 = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rm, so4, 0, 2));
        const f32x4_t t0 = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rv, so, 0, 2));
        const f32x4_t t1 = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rv, so4, 0, 2));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            sm[e] = s0[e]; sm[e + 4] = s1[e];
            sv[e] = t0[e]; sv[e + 4] = t1[e];
        }
    }

    static __device__ __forceinline__ float code_at(u32x2_t c, int e)
    {
        // sign-extend byte e of the 8 packed codes
        const uint32_t word = c[e >> 2];
        return (float)((int32_t)(word << (24 - 8 * (e & 3))) >> 24);
    }

    __device__ __forceinline__ void state_at(const Args &a, int i, const float *g, int e,
                                             float &w1, float &m1, float &v1, float &rv1) const
    {
        const float m0 = sm[e] * code_at(pm[i], e);
        const float r0 = sv[e] * code_at(pv[i], e);
        const float w0 = (e & 1) ? bf_hi(pw[i][e >> 1]) : bf_lo(pw[i][e >> 1]);
        adamw_elem(g[e], w0, m0, r0 * r0, a.h, w1, m1, v1, rv1);
    }

    // Contains one LDS barrier (the cross-wave absmax), which every wave of the
    // workgroup must also execute.
    __device__ __forceinline__ void run(const Args &a, int p0, int q0, int s, const float *Gs,
                                        float *red)
    {
        const int rs = s / M::LPR, qo = (s % M::LPR) * 8, q = q0 + qo;
        const bool qok = q < a.d_in;
        float am[8], av[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) am[e] = av[e] = 0.0f;

        // pass 1: weight update (from the unquantised fp32 state) and block absmax
#pragma unroll
        for (int i = 0; i < M::NPASS; ++i) {
            const int p = p0 + i * M::RPP + rs;
            const float *gr = Gs + (i * M::RPP + rs) * M::GP + qo;
            const f32x4_t g0 = *reinterpret_cast<const f32x4_t *>(gr);
            const f32x4_t g1 = *reinterpret_cast<const f32x4_t *>(gr + 4);
            const float g[8] = {g0[0], g0[1], g0[2], g0[3], g1[0], g1[1], g1[2], g1[3]};
            float wo[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                float m1, v1, rv1;
                state_at(a, i, g, e, wo[e], m1, v1, rv1);
                am[e] = fmaxf(am[e], fabsf(m1));
                av[e] = fmaxf(av[e], rv1);
            }
            if (qok && p < a.d_out) {
                u32x4_t wn;
#pragma unroll
                for (int k = 0; k < 4; ++k) wn[k] = pack_bf16(wo[2 * k], wo[2 * k + 1]);
                st_nt<u32x4_t>(a.W + (size_t)p * a.d_in + q, wn);
            }
            // close this pass's absmax now: otherwise the compiler keeps every pass's m' and
            // sqrt(v') live to combine them after the loop (200 VGPRs instead of ~100)
#pragma unroll
            for (int e = 0; e < 8; ++e) asm volatile("" : "+v"(am[e]), "+v"(av[e]));
            __builtin_amdgcn_sched_barrier(0);
        }
        // lanes of one wave sharing these columns differ in the bits above log2(LPR)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
#pragma unroll
            for (int d = M::LPR; d < 64; d <<= 1) {
                am[e] = fmaxf(am[e], __shfl_xor(am[e], d));
                av[e] = fmaxf(av[e], __shfl_xor(av[e], d));
            }
        }
        const int sw = s >> 6;
        if ((s & 63) < M::LPR) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                red[sw * BQ + qo + e] = am[e];
                red[4 * BQ + sw * BQ + qo + e] = av[e];
            }
        }
        lds_barrier();
        // new scales: s = absmax / 127 (fp32, correctly rounded); kept as reciprocals
        float rcm[8], rcv[8];
        {
            float scm[8], scv[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                float xm = red[qo + e], xv = red[4 * BQ + qo + e];
#pragma unroll
                for (int w = 1; w < 4; ++w) {
                    xm = fmaxf(xm, red[w * BQ + qo + e]);
                    xv = fmaxf(xv, red[4 * BQ + w * BQ + qo + e]);
                }
                scm[e] = xm / 127.0f;
                scv[e] = xv / 127.0f;
                rcm[e] = scm[e] > 0.0f ? __builtin_amdgcn_rcpf(scm[e]) : 0.0f;
                rcv[e] = scv[e] > 0.0f ? __builtin_amdgcn_rcpf(scv[e]) : 0.0f;
            }
            // every lane read its old scales before pass 1, i.e. before the barrier above
            if (rs == 0 && qok) {
                const size_t so = (size_t)(p0 / I8_BLOCK) * a.d_in + q;
                st_nt<f32x4_t>(a.ms + so, f32x4_t{scm[0], scm[1], scm[2], scm[3]});
                st_nt<f32x4_t>(a.ms + so + 4, f32x4_t{scm[4], scm[5], scm[6], scm[7]});
                st_nt<f32x4_t>(a.vs + so, f32x4_t{scv[0], scv[1], scv[2], scv[3]});
                st_nt<f32x4_t>(a.vs + so + 4, f32x4_t{scv[4], scv[5], scv[6], scv[7]});
            }
        }
        // pass 2: re-quantise.  Hide the prefetched state from common-subexpression
        // elimination so that pass 2 recomputes m' and sqrt(v') (bit-identical, same
        // instructions) instead of keeping 64 pass-1 intermediates alive.
#pragma unroll
        for (int i = 0; i < M::NPASS; ++i) {
            asm volatile("" : "+v"(pm[i]));
            asm volatile("" : "+v"(pv[i]));
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            asm volatile("" : "+v"(sm[e]));
            asm volatile("" : "+v"(sv[e]));
        }
#pragma unroll
        for (int i = 0; i < M::NPASS; ++i) {
            const int p = p0 + i * M::RPP + rs;
            const float *gr = Gs + (i * M::RPP + rs) * M::GP + qo;
            const f32x4_t g0 = *reinterpret_cast<const f32x4_t *>(gr);
            const f32x4_t g1 = *reinterpret_cast<const f32x4_t *>(gr + 4);
            const float g[8] = {g0[0], g0[1], g0[2], g0[3], g1[0], g1[1], g1[2], g1[3]};
            uint32_t cm[2] = {0u, 0u}, cv[2] = {0u, 0u};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                float w1, m1, v1, rv1;
                state_at(a, i, g, e, w1, m1, v1, rv1);
                const float qm = fminf(fmaxf(__builtin_rintf(m1 * rcm[e]), -127.0f), 127.0f);
                float qv = fminf(fmaxf(__builtin_rintf(rv1 * rcv[e]), 1.0f), 127.0f);
                if (!(rcv[e] > 0.0f)) qv = 0.0f;
                cm[e >> 2] |= ((uint32_t)(int32_t)qm & 0xFFu) << (8 * (e & 3));
                cv[e >> 2] |= ((uint32_t)(int32_t)qv & 0xFFu) << (8 * (e & 3));
            }
            if (qok && p < a.d_out) {
                const size_t off = (size_t)p * a.d_in + q;
                st_nt<u32x2_t>(static_cast<int8_t *>(a.m) + off, u32x2_t{cm[0], cm[1]});
                st_nt<u32x2_t>(static_cast<int8_t *>(a.v) + off, u32x2_t{cv[0], cv[1]});
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    }
};

// Store G (the two-kernel path's GEMM epilogue), bf16 (round to nearest even) or fp32.
template <int BP, int BQ, bool F32>
__device__ __forceinline__ void epi_store_g(const Args &a, int p0, int q0, int s, const float *Gs)
{
    using M = EpiMap<BP, BQ>;
    const int rs = s / M::LPR, qo = (s % M::LPR) * 8, q = q0 + qo;
#pragma unroll
    for (int i = 0; i < M::NPASS; ++i) {
        const int p = p0 + i * M::RPP + rs;
        if (!(q < a.d_in && p < a.d_out)) continue;
        const float *gr = Gs + (i * M::RPP + rs) * M::GP + qo;
        const f32x4_t g0 = *reinterpret_cast<const f32x4_t *>(gr);
        const f32x4_t g1 = *reinterpret_cast<const f32x4_t *>(gr + 4);
        const size_t off = (size_t)p * a.d_in + q;
        if constexpr (F32) {
            st_nt<f32x4_t>(static_cast<float *>(a.G) + off, g0);
            st_nt<f32x4_t>(static_cast<float *>(a.G) + off + 4, g1);
        } else {
            u32x4_t o = {pack_bf16(g0[0], g0[1]), pack_bf16(g0[2], g0[3]),
                         pack_bf16(g1[0], g1[1]), pack_bf16(g1[2], g1[3])};
            st_nt<u32x4_t>(static_cast<uint16_t *>(a.G) + off, o);
        }
    }
}

// ------------------------------------------------------------------------ kernels

// At most 128 VGPRs (four waves per SIMD): two 512-thread workgroups per CU, one math and
// one stream wave of each on every SIMD.  At 129-136 registers only one would fit.
template <int BP, int BQ, int MK, int EPI, int AH = 0>
__global__ void __launch_bounds__(NT, 4) fused_kernel(GroupArgs g)
{
    static_assert(MK != MK_I8, "int8 moments run in pipelined_i8_kernel");
    static_assert(MK != MK_I8R64 || EPI == EPI_ADAMW || EPI == EPI_STORE_BF16 || EPI == EPI_STORE_F32,
                  "row-block int8 moments: AdamW only");
    static_assert(MK != MK_FP8 || EPI == EPI_ADAMW || EPI == EPI_ADAMW_WFP8, "fp8 moments: AdamW only");
    static_assert(EPI != EPI_ADAMW_WFP8 || MK == MK_BF16 || MK == MK_FP8, "fp8 weights: bf16 or fp8 moments");
    using ML = Mainloop<BP, BQ, NSTAGE, TK128>;
    using EM = EpiMap<BP, BQ>;
    constexpr int MAIN = ML::LDS_BYTES > EM::GS_BYTES ? ML::LDS_BYTES : EM::GS_BYTES;
    __shared__ __attribute__((aligned(16))) unsigned char smem[MAIN];
    float *Gs = reinterpret_cast<float *>(smem);

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int s = tid - NROLE;
    // This workgroup's tile: XCD-aware over all tiles of the group, then the matrix that
    // owns it and the tile's place in that matrix.
    const int t = xcd_remap(blockIdx.x, g.start[g.n]);
    int mi = 0;
    while (mi + 1 < g.n && t >= g.start[mi + 1]) ++mi;
    const Args a = g.a[mi];
    constexpr bool LEAD = EPI != EPI_STORE_BF16 && EPI != EPI_STORE_F32;
    const int nbar = ML::nbar(a.T, LEAD);
    int tp, tq;
    raster(t - g.start[mi], a.tiles_p, a.tiles_q, a.group_p, tp, tq);
    const int p0 = tp * BP, q0 = tq * BQ;
    if (wave < 4) {
        ML ml;
        ml.run(a, p0, q0, smem, wave, lane, LEAD);
        ml.template stage_g<EM::GP>(Gs, wave, lane);
        lds_barrier();
    } else if constexpr (EPI != EPI_STORE_BF16 && EPI != EPI_STORE_F32) {
        typename EpiSel<BP, BQ, MK, EPI, AH>::T ep;
        if constexpr (IsEpiQ<decltype(ep)>::value) ep.first_tile = (t == g.start[mi]);
        // The state prefetch leaves after the mainloop's first barrier (its first chunks'
        // DMA is then ahead of it); for the int8 row-block state, after the barriers of two
        // more chunks.  Measured at T = 512: the Llama-3.1-8B sweep 19.54-19.55 against
        // 19.66 ms with the prefetch issued as the workgroup starts, the MLP with int8 row
        // blocks 0.430 against 0.438 ms; later issue was slower for bf16 state.
        constexpr int PF_AT = MK == MK_I8R64 ? 3 : 1;
        int done = 0;
        for (; done < PF_AT && done < nbar; ++done) lds_barrier();
        ep.prefetch(a, p0, q0, s);
        for (; done < nbar; ++done) lds_barrier();
        lds_barrier();
        ep.run(a, p0, q0, s, Gs);
    } else {
        for (int i = 0; i < nbar; ++i) lds_barrier();
        lds_barrier();
        epi_store_g<BP, BQ, EPI == EPI_STORE_F32>(a, p0, q0, s, Gs);
    }
}

template <int BP, int BQ, int MK, bool GF32>
__global__ void __launch_bounds__(NROLE, 2) adamw_kernel(Args a)
{
    using EM = EpiMap<BP, BQ>;
    constexpr int RED = (MK == MK_I8) ? 2 * 4 * BQ * 4 : 0;
    __shared__ __attribute__((aligned(16))) unsigned char smem[EM::GS_BYTES + RED];
    float *Gs = reinterpret_cast<float *>(smem);
    float *red = reinterpret_cast<float *>(smem + EM::GS_BYTES);
    const int s = threadIdx.x;
    int tp, tq;
    tile_of(blockIdx.x, gridDim.x, a.tiles_p, a.tiles_q, a.group_p, tp, tq);
    const int p0 = tp * BP, q0 = tq * BQ;

    auto stage = [&]() {
        const int rs = s / EM::LPR, qo = (s % EM::LPR) * 8, q = q0 + qo;
#pragma unroll
        for (int i = 0; i < EM::NPASS; ++i) {
            const int p = p0 + i * EM::RPP + rs;
            f32x4_t g0 = {0, 0, 0, 0}, g1 = g0;
            if (q < a.d_in && p < a.d_out) {
                const size_t off = (size_t)p * a.d_in + q;
                if constexpr (GF32) {
                    g0 = ld_nt<f32x4_t>(static_cast<const float *>(a.G) + off);
                    g1 = ld_nt<f32x4_t>(static_cast<const float *>(a.G) + off + 4);
                } else {
                    const u32x4_t b = ld_nt<u32x4_t>(static_cast<const uint16_t *>(a.G) + off);
                    g0 = f32x4_t{bf_lo(b[0]), bf_hi(b[0]), bf_lo(b[1]), bf_hi(b[1])};
                    g1 = f32x4_t{bf_lo(b[2]), bf_hi(b[2]), bf_lo(b[3]), bf_hi(b[3])};
                }
            }
            float *gr = Gs + (i * EM::RPP + rs) * EM::GP + qo;
            *reinterpret_cast<f32x4_t *>(gr) = g0;
            *reinterpret_cast<f32x4_t *>(gr + 4) = g1;
        }
    };
    if constexpr (MK == MK_I8) {
        EpiAdamWI8<BP, BQ> ep;
        ep.prefetch(a, p0, q0, s);
        stage();
        lds_barrier();
        ep.run(a, p0, q0, s, Gs, red);
    } else {
        static_assert(MK != MK_FP8, "fp8 moments are stepped by the fused kernel only");
        typename EpiSel<BP, BQ, MK, EPI_ADAMW>::T ep;
        ep.prefetch(a, p0, q0, s);
        stage();
        lds_barrier();
        ep.run(a, p0, q0, s, Gs);
    }
}

// ------------------------------------------------ int8 moments: tiles pipelined per CU
//
// One workgroup per CU steps a sequence of 256x64 tiles.  Its four math waves run the
// mainloop of tile k while its stream waves finish tile k-1 (App. B update of W, block
// absmax, re-quantisation of m and sqrt(v)) and load tile k's state for the next period.
// G reaches the stream waves through an LDS stage of its own, written by the math waves
// between the barriers H1 and H2 that close each period and read by the stream waves
// during the next period, before its H1; pass 1 leaves m' in that stage in place of g for
// pass 2.  Every workgroup barrier is executed by all waves: a period has nb = max(nch, 2)
// barriers (the mainloop's chunk barriers, padded), then H1 and H2.

template <int NSW>
struct StreamI8 {
    using M = EpiMap<BP_I8, BQ_I8, NSW * 64>;           // 8 lanes per row, 8*NSW rows per pass
    static constexpr int NPASS = M::NPASS;
    u32x4_t w[NPASS];                                   // W row of each pass (8 bf16)
    u32x2_t cm[NPASS], cv[NPASS];                       // m and sqrt(v) codes (8 int8 each)
    float sm[8], sv[8];                                 // the block's old scales of this lane's columns
    float am[8], av[8];                                 // absmax partials
    float rv[NPASS][8];                                 // sqrt(v') of each pass, for pass 2
    float rcm[8], rcv[8];                               // reciprocals of the new scales
    float lov[8];                                       // least sqrt(v) code: 1, or 0 in an all-zero block

    // Loads of the state of tile (p0, q0) of matrix a: row I of every pass, then the scales.
    template <int I>
    __device__ __forceinline__ void load_w(const Args &a, int p0, int q0, int s)
    {
        const int p = p0 + I * M::RPP + s / M::LPR, q = q0 + (s % M::LPR) * 8;
        const __amdgpu_buffer_rsrc_t r = rsrc_of(a.W, 2ull * (uint64_t)a.d_out * (uint64_t)a.d_in);
        w[I] = __builtin_amdgcn_raw_buffer_load_b128(r, elem_off(p, q, a.d_out, a.d_in, 2), 0, 2);
    }
    template <int I>
    __device__ __forceinline__ void load_codes(const Args &a, int p0, int q0, int s)
    {
        const int p = p0 + I * M::RPP + s / M::LPR, q = q0 + (s % M::LPR) * 8;
        const uint64_t n = (uint64_t)a.d_out * (uint64_t)a.d_in;
        const uint32_t off = elem_off(p, q, a.d_out, a.d_in, 1);
        // Plain (not non-temporal) loads: a tile's 64-byte code rows are half of a 128-byte
        // line whose other half the neighbouring tile reads a little later from L2 (mlp_i8:
        // 314 instead of 334 MB fetched per launch).
        cm[I] = __builtin_amdgcn_raw_buffer_load_b64(rsrc_of(a.m, n), off, 0, 0);
        cv[I] = __builtin_amdgcn_raw_buffer_load_b64(rsrc_of(a.v, n), off, 0, 0);
    }
    __device__ __forceinline__ void load_scales(const Args &a, int p0, int q0, int s)
    {
        const int q = q0 + (s % M::LPR) * 8, blk = p0 / I8_BLOCK, nblk = (a.d_out + I8_BLOCK - 1) / I8_BLOCK;
        const uint64_t n = 4ull * (uint64_t)nblk * (uint64_t)a.d_in;
        const uint32_t off = elem_off(blk, q, nblk, a.d_in, 4);
        const __amdgpu_buffer_rsrc_t rm = rsrc_of(a.ms, n), rv = rsrc_of(a.vs, n);
        const f32x4_t s0 = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rm, off, 0, 2));
        const f32x4_t s1 = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rm, off + 16u, 0, 2));
        const f32x4_t t0 = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rv, off, 0, 2));
        const f32x4_t t1 = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rv, off + 16u, 0, 2));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            sm[e] = s0[e]; sm[e + 4] = s1[e];
            sv[e] = t0[e]; sv[e + 4] = t1[e];
        }
    }
    template <int I = 0>
    __device__ __forceinline__ void load_all(const Args &a, int p0, int q0, int s)
    {
        load_w<I>(a, p0, q0, s);
        load_codes<I>(a, p0, q0, s);
        if constexpr (I + 1 < NPASS) load_all<I + 1>(a, p0, q0, s);
        else load_scales(a, p0, q0, s);
    }

    // Wait once for the slot's loads (issued a period earlier, so long done), then hide
    // the registers from the compiler's wait tracking: what follows does not wait for the
    // stores of the previous tile.
    __device__ __forceinline__ void settle()
    {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
        for (int i = 0; i < NPASS; ++i) asm volatile("" : "+v"(w[i]), "+v"(cm[i]), "+v"(cv[i]));
#pragma unroll
        for (int e = 0; e < 8; ++e) asm volatile("" : "+v"(sm[e]), "+v"(sv[e]));
    }

    __device__ __forceinline__ void reset()
    {
#pragma unroll
        for (int e = 0; e < 8; ++e) am[e] = av[e] = 0.0f;
    }

    // G of row I of this lane (8 columns) from the LDS stage.
    template <int I>
    static __device__ __forceinline__ void g_row(const float *Gs, int s, float g[8])
    {
        const float *gr = Gs + (I * M::RPP + s / M::LPR) * M::GP + (s % M::LPR) * 8;
        const f32x4_t g0 = *reinterpret_cast<const f32x4_t *>(gr);
        const f32x4_t g1 = *reinterpret_cast<const f32x4_t *>(gr + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            g[e] = g0[e];
            g[e + 4] = g1[e];
        }
    }

    // m' of row I of this lane back into the LDS stage, over its g.
    template <int I>
    static __device__ __forceinline__ void put_row(float *Gs, int s, const float x[8])
    {
        float *gr = Gs + (I * M::RPP + s / M::LPR) * M::GP + (s % M::LPR) * 8;
        *reinterpret_cast<f32x4_t *>(gr) = f32x4_t{x[0], x[1], x[2], x[3]};
        *reinterpret_cast<f32x4_t *>(gr + 4) = f32x4_t{x[4], x[5], x[6], x[7]};
    }

    // The element's state before and after the step (App. B: m = s_m q_m, v = (s_v q_v)^2).
    __device__ __forceinline__ void state_at(const Hyper &h, int i, float g, int e, float &w1, float &m1,
                                             float &v1, float &rv1) const
    {
        const float m0 = sm[e] * EpiAdamWI8<BP_I8, BQ_I8>::code_at(cm[i], e);
        const float r0 = sv[e] * EpiAdamWI8<BP_I8, BQ_I8>::code_at(cv[i], e);
        const float w0 = (e & 1) ? bf_hi(w[i][e >> 1]) : bf_lo(w[i][e >> 1]);
        adamw_elem(g, w0, m0, r0 * r0, h, w1, m1, v1, rv1);
    }

    // Pass 1, row I of tile (p0, q0), from the unquantised fp32 state: W' is stored, m'
    // replaces g in the LDS stage and sqrt(v') stays in registers, both waiting for the
    // block's new scales; absmax partials.  The row's W and code registers are then free
    // and take row I of the next tile (pn, qn) of matrix an, and after the last row the
    // scale registers take that tile's scales.
    template <int I>
    __device__ __forceinline__ void pass1(const Args &a, int p0, int q0, int s, float *Gs,
                                          const Args &an, int pn, int qn, bool refill)
    {
        const int p = p0 + I * M::RPP + s / M::LPR, q = q0 + (s % M::LPR) * 8;
        float g[8], wo[8], mo[8];
        g_row<I>(Gs, s, g);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            float v1;
            state_at(a.h, I, g[e], e, wo[e], mo[e], v1, rv[I][e]);
            am[e] = fmaxf(am[e], fabsf(mo[e]));
            av[e] = fmaxf(av[e], rv[I][e]);
        }
        put_row<I>(Gs, s, mo);
        if (p < a.d_out && q < a.d_in) {
            u32x4_t wn;
#pragma unroll
            for (int k = 0; k < 4; ++k) wn[k] = pack_bf16(wo[2 * k], wo[2 * k + 1]);
            st_nt<u32x4_t>(a.W + (size_t)p * a.d_in + q, wn);
        }
        asm volatile("" ::"v"(w[I]), "v"(cm[I]), "v"(cv[I]));
        if (refill) {
            load_w<I>(an, pn, qn, s);
            load_codes<I>(an, pn, qn, s);
            if constexpr (I + 1 == NPASS) {
#pragma unroll
                for (int e = 0; e < 8; ++e) asm volatile("" ::"v"(sm[e]), "v"(sv[e]));
                load_scales(an, pn, qn, s);
            }
        }
    }

    // Max of x >= 0 over the 8 lanes l, l^8, ..., l^56 that hold the same columns (a wave's 8 rows):
    // a DPP rotation by 8 within each row of 16 lanes, then the CDNA4 lane swaps of rows
    // 2k with 2k+1 and of the two halves of the wave.
    static __device__ __forceinline__ float max_rows(float x)
    {
        static_assert(M::LPR == 8, "8 lanes per row");
        int b = __float_as_int(x);
        b = max(b, dpp_i<0x128>(b));
        const auto h = __builtin_amdgcn_permlane16_swap(b, b, false, false);
        b = max((int)h[0], (int)h[1]);
        const auto w = __builtin_amdgcn_permlane32_swap(b, b, false, false);
        return __int_as_float(max((int)w[0], (int)w[1]));
    }

    // Block absmax of this lane's columns over its rows: within the wave, then (through
    // LDS, across the barrier that follows) across the NSW stream waves.
    __device__ __forceinline__ void partials(int s, float *red)
    {
        const int qo = (s % M::LPR) * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            am[e] = max_rows(am[e]);
            av[e] = max_rows(av[e]);
        }
        const int sw = s >> 6;
        if ((s & 63) < M::LPR) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                red[sw * BQ_I8 + qo + e] = am[e];
                red[NSW * BQ_I8 + sw * BQ_I8 + qo + e] = av[e];
            }
        }
    }

    // After the barrier: the block's new scales s = absmax / 127, one per thread of the
    // first 2*BQ (m for the first BQ columns, sqrt(v) for the next): the column's absmax
    // over the stream waves' partials; s is stored and its reciprocal put in LDS.
    __device__ __forceinline__ void scales(const Args &a, int p0, int q0, int s, float *red)
    {
        if (s < 2 * BQ_I8) {
            const int kind = s / BQ_I8, c = s % BQ_I8;
            const float *r = red + kind * NSW * BQ_I8 + c;
            float x = r[0];
#pragma unroll
            for (int wv = 1; wv < NSW; ++wv) x = fmaxf(x, r[wv * BQ_I8]);
            const float sc = x / 127.0f;
            red[2 * NSW * BQ_I8 + s] = sc > 0.0f ? __builtin_amdgcn_rcpf(sc) : 0.0f;
            if (q0 + c < a.d_in) {
                float *dst = kind ? a.vs : a.ms;
                st_nt<float>(dst + (size_t)(p0 / I8_BLOCK) * a.d_in + q0 + c, sc);
            }
        }
    }

    // After the next barrier: the reciprocals of this lane's eight columns.
    __device__ __forceinline__ void recips(int s, const float *red)
    {
        const float *r = red + 2 * NSW * BQ_I8 + (s % M::LPR) * 8;
        const f32x4_t m0 = *reinterpret_cast<const f32x4_t *>(r);
        const f32x4_t m1 = *reinterpret_cast<const f32x4_t *>(r + 4);
        const f32x4_t v0 = *reinterpret_cast<const f32x4_t *>(r + BQ_I8);
        const f32x4_t v1 = *reinterpret_cast<const f32x4_t *>(r + BQ_I8 + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            rcm[e] = m0[e]; rcm[e + 4] = m1[e];
            rcv[e] = v0[e]; rcv[e + 4] = v1[e];
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) lov[e] = rcv[e] > 0.0f ? 1.0f : 0.0f;
    }

    // Pass 2, row I: m' (from the LDS stage) and sqrt(v') (from registers) quantised
    // against the new scales (v codes at least 1 in a non-zero block); the codes are stored.
    template <int I>
    __device__ __forceinline__ void pass2(const Args &a, int p0, int q0, int s, const float *Gs)
    {
        const int p = p0 + I * M::RPP + s / M::LPR, q = q0 + (s % M::LPR) * 8;
        float ym[8], yv[8];
        g_row<I>(Gs, s, ym);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            ym[e] *= rcm[e];
            yv[e] = rv[I][e] * rcv[e];
        }
        const u32x2_t qm = pack_codes(ym, -127.0f), qv = pack_codes(yv, lov);
        if (p < a.d_out && q < a.d_in) {
            const size_t off = (size_t)p * a.d_in + q;
            st_nt<u32x2_t>(static_cast<int8_t *>(a.m) + off, qm);
            st_nt<u32x2_t>(static_cast<int8_t *>(a.v) + off, qv);
        }
    }

    // The whole epilogue of one tile, spread over nb >= 2 barriers: pass-1 rows over the
    // first half (its last barrier, A, separates the absmax partials from their reads), the
    // scales between A and the next barrier B, pass-2 rows over the rest.  Executes exactly
    // nb barriers.
    template <int I = 0>
    __device__ __forceinline__ void p1_all(const Args &a, int p0, int q0, int s, float *Gs,
                                           const Args &an, int pn, int qn, bool refill, int half, int &done,
                                           float *red)
    {
        pass1<I>(a, p0, q0, s, Gs, an, pn, qn, refill);
        if constexpr (I + 1 < NPASS) {
            for (const int t = ((I + 1) * half) / NPASS; done < t && done < half - 1; ++done) lds_barrier();
            p1_all<I + 1>(a, p0, q0, s, Gs, an, pn, qn, refill, half, done, red);
        } else {
            for (; done < half - 1; ++done) lds_barrier();
            partials(s, red);
            lds_barrier();                                   // A
            ++done;
        }
    }
    template <int I = 0>
    __device__ __forceinline__ void p2_all(const Args &a, int p0, int q0, int s, const float *Gs, int half,
                                           int nb, int &done)
    {
        pass2<I>(a, p0, q0, s, Gs);
        const int t = half + 1 + ((I + 1) * (nb - half - 1)) / NPASS;
        for (; done < t; ++done) lds_barrier();
        if constexpr (I + 1 < NPASS) p2_all<I + 1>(a, p0, q0, s, Gs, half, nb, done);
    }
    // G of the tile stays in its LDS stage (m' after pass 1) until this returns (the math
    // waves overwrite it only after the next H1).
    __device__ __forceinline__ void tile(const Args &a, int p0, int q0, int s, float *Gs,
                                         const Args &an, int pn, int qn, bool refill, int nb, float *red)
    {
        const int half = nb / 2;
        int done = 0;
        reset();
        p1_all(a, p0, q0, s, Gs, an, pn, qn, refill, half, done, red);
        scales(a, p0, q0, s, red);
        lds_barrier();                                       // B
        ++done;
        recips(s, red);
        p2_all(a, p0, q0, s, Gs, half, nb, done);
    }
};

constexpr int NSW_I8P = FORGE_NSW_I8P;                  // stream waves of the pipelined int8 kernel
constexpr int NT_I8P = NROLE + NSW_I8P * 64;

__global__ void __launch_bounds__(NT_I8P, NT_I8P / 256) pipelined_i8_kernel(GroupArgs g)
{
    using ML = Mainloop<BP_I8, BQ_I8, NS_I8P, 32>;
    using EM = EpiMap<BP_I8, BQ_I8, NSW_I8P * 64>;
    constexpr int RED_BYTES = (2 * NSW_I8P * BQ_I8 + 2 * BQ_I8) * 4;   // absmax partials, then reciprocals
    __shared__ __attribute__((aligned(16))) unsigned char smem[EM::GS_BYTES + ML::LDS_BYTES + RED_BYTES];
    float *Gs = reinterpret_cast<float *>(smem);
    unsigned char *ring = smem + EM::GS_BYTES;
    float *red = reinterpret_cast<float *>(smem + EM::GS_BYTES + ML::LDS_BYTES);

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int total = g.start[g.n];
    const int K = (total - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x;   // tiles of this workgroup
    // tile k of this workgroup: its matrix and origin
    auto locate = [&](int k, int &mi, int &p0, int &q0) {
        const int t = xcd_remap((int)blockIdx.x + k * (int)gridDim.x, total);
        mi = 0;
        while (mi + 1 < g.n && t >= g.start[mi + 1]) ++mi;
        int tp, tq;
        raster(t - g.start[mi], g.a[mi].tiles_p, g.a[mi].tiles_q, g.a[mi].group_p, tp, tq);
        p0 = tp * BP_I8;
        q0 = tq * BQ_I8;
    };
    const int nch = ML::nch(g.a[0].T);
    const int nb = nch > 2 ? nch : 2;

    if (wave < 4) {
        ML ml;
        int mi, p0, q0;
        locate(0, mi, p0, q0);
        ml.begin(g.a[mi], p0, q0, ring, wave, lane);
        for (int k = 0; k < K; ++k) {
            ml.body(g.a[mi], ring, wave);
            for (int c = nch; c < nb; ++c) lds_barrier();
            lds_barrier();                                   // H1: the stream waves hold G(k-1)
            ml.template stage_g<EM::GP>(Gs, wave, lane);
            if (k + 1 < K) {
                locate(k + 1, mi, p0, q0);
                ml.begin(g.a[mi], p0, q0, ring, wave, lane);
            }
            lds_barrier();                                   // H2: G(k) is in LDS
        }
        // the stream waves finish the last tile with nb more barriers
        for (int c = 0; c < nb; ++c) lds_barrier();
        return;
    }

    const int s = tid - NROLE;
    StreamI8<NSW_I8P> st;
    int mp, pp, qp;                                          // the tile whose state is in the slot
    locate(0, mp, pp, qp);
    st.load_all(g.a[mp], pp, qp, s);
    for (int c = 0; c < nb; ++c) lds_barrier();              // period 0: nothing to finish yet
    lds_barrier();                                           // H1
    lds_barrier();                                           // H2
    for (int k = 1; k <= K; ++k) {
        // finish tile k-1; during it, load tile k's state (for the next period)
        st.settle();
        int mk = mp, pk = pp, qk = qp;
        const bool more = k < K;
        if (more) locate(k, mk, pk, qk);
        st.tile(g.a[mp], pp, qp, s, Gs, g.a[mk], pk, qk, more, nb, red);
        if (more) {
            lds_barrier();                                   // H1
            lds_barrier();                                   // H2
        }
        mp = mk;
        pp = pk;
        qp = qk;
    }
}

// ------------------------------------------------------------------------ launchers

TileShape tile_shape(int mk)
{
    if (mk == MK_I8) return TileShape{BP_I8, BQ_I8, 32};
    return TileShape{BP_F, BQ_F, TK128};
}

// Tile rows per raster group, by the shape of the tile grid (measured on the Llama-3.1-8B
// shapes at T = 512): matrices wider than tall walk 24 rows at a time, very tall ones 8,
// the rest 16.  The 64 tiles resident on an XCD then span a few hundred KB of operand
// slabs in its L2 and a few thousand rows of the state, in runs of 0.7-2 KB per row.
static int raster_rows(int tiles_p, int tiles_q)
{
    if (tiles_q > tiles_p) return 24;
    if (tiles_p > 16 * tiles_q) return 8;
    return 16;
}

static Args with_grid(Args a, int bp, int bq, int &ntiles, int group_p = 0)
{
    a.tiles_p = (a.d_out + bp - 1) / bp;
    a.tiles_q = (a.d_in + bq - 1) / bq;
    a.group_p = group_p ? group_p : FORGE_GROUP_P ? FORGE_GROUP_P : raster_rows(a.tiles_p, a.tiles_q);
    ntiles = a.tiles_p * a.tiles_q;
    return a;
}

// Tile grid of each matrix, prefix sums of their tile counts, and the launch.
template <int BP, int BQ, int MK, int EPI>
static hipError_t launch_group(const Args *a, int n, hipStream_t st)
{
    GroupArgs g;
    g.n = n;
    g.start[0] = 0;
    for (int i = 0; i < n; ++i) {
        int nt;
        // int8 row-block state: groups of 8 tile rows (measured on the MLP projections at
        // T = 512: 5 % faster than the shape rule, whose 24-row groups suit bf16 state)
        g.a[i] = with_grid(a[i], BP, BQ, nt, MK == MK_I8R64 ? 8 : 0);
        g.start[i + 1] = g.start[i] + nt;
    }
    for (int i = n; i < MAX_GROUP; ++i) {
        g.a[i] = g.a[0];
        g.start[i + 1] = g.start[n];
    }
    if (g.start[n] == 0) return hipSuccess;
    // Prefetch depth by launch length (AdamW on bf16 state): a launch of at least 8 waves of
    // resident tiles, or with a long token loop (T >= 1024 in every matrix), loads all eight
    // row passes of a tile's state during its mainloop, a shorter one six.  Measured per
    // launch group of the Llama-3.1-8B sweep at T = 512: lm_head (63 waves) 1157 against
    // 1222 us, gate+up (14) even, down (7), o (2) and q+k+v (3) 1-7 % slower with eight; on
    // 4096 x 4096 over three rotated copies, eight were 2-4.5 % faster at T = 1024-4096
    // (T = 4096: 145.9-146.4 against 148.9-149.1 us).
    int min_t = a[0].T;
    for (int i = 1; i < n; ++i) min_t = a[i].T < min_t ? a[i].T : min_t;
    if constexpr (MK == MK_BF16 && EPI == EPI_ADAMW)
        if (g.start[n] >= 8 * 2 * device_cu_count() || min_t >= 1024) {
            hipLaunchKernelGGL((fused_kernel<BP, BQ, MK, EPI, 8>), dim3(g.start[n]), dim3(NT), 0, st, g);
            return hipGetLastError();
        }
    hipLaunchKernelGGL((fused_kernel<BP, BQ, MK, EPI>), dim3(g.start[n]), dim3(NT), 0, st, g);
    return hipGetLastError();
}

int device_cu_count()
{
    static std::mutex mu;
    static int known[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    std::lock_guard<std::mutex> lock(mu);
    if (known[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
        known[dev] = n;
    }
    return known[dev];
}

// Raster rows of the pipelined int8 kernel: the 32 tiles resident on an XCD walk the
// columns of a group of tile rows, so the group's dY slabs (T x 256 bf16 each) are read
// from HBM once and then served by the XCD's 4 MB L2.  Groups are kept to about 2 MB of
// dY (8 rows at T = 512; the 24 rows chosen for 128x128 tiles span 6 MB there, and
// the kernel fetched 3.8x its algorithmic reads, against 1.33x with 8).
static int raster_rows_i8(int T)
{
    if (FORGE_GROUP_P_I8) return FORGE_GROUP_P_I8;
    const long slab = (long)T * BP_I8 * 2;
    int g = 8;
    while (g > 1 && g * slab > (2l << 20)) g >>= 1;
    return g;
}

// int8 moments: one persistent workgroup per CU, tiles pipelined (pipelined_i8_kernel).
static hipError_t launch_i8_pipelined(const Args *a, int n, hipStream_t st)
{
    GroupArgs g;
    g.n = n;
    g.start[0] = 0;
    for (int i = 0; i < n; ++i) {
        int nt;
        g.a[i] = with_grid(a[i], BP_I8, BQ_I8, nt, raster_rows_i8(a[i].T));
        g.start[i + 1] = g.start[i] + nt;
    }
    for (int i = n; i < MAX_GROUP; ++i) {
        g.a[i] = g.a[0];
        g.start[i + 1] = g.start[n];
    }
    const int total = g.start[n];
    if (total == 0) return hipSuccess;
    const int ncu = device_cu_count();
    const int grid = total < ncu ? total : ncu;
    hipLaunchKernelGGL(pipelined_i8_kernel, dim3(grid), dim3(NT_I8P), 0, st, g);
    return hipGetLastError();
}

hipError_t launch_fused_group(const Args *a, int n, int mk, hipStream_t st)
{
    if (mk == MK_I8) return launch_i8_pipelined(a, n, st);
    if (mk == MK_I8R64) return launch_group<BP_F, BQ_F, MK_I8R64, EPI_ADAMW>(a, n, st);
    if (mk == MK_FP8) return launch_group<BP_F, BQ_F, MK_FP8, EPI_ADAMW>(a, n, st);
    if (mk == MK_BF16) return launch_group<BP_F, BQ_F, MK_BF16, EPI_ADAMW>(a, n, st);
    return launch_group<BP_F, BQ_F, MK_F32, EPI_ADAMW>(a, n, st);
}

template <int E>
static hipError_t launch_rule(const Args *a, int n, int mk, hipStream_t st)
{
    if (mk == MK_BF16) return launch_group<BP_F, BQ_F, MK_BF16, E>(a, n, st);
    return launch_group<BP_F, BQ_F, MK_F32, E>(a, n, st);
}

hipError_t launch_fused_rule(const Args *a, int n, int epi, int mk, hipStream_t st)
{
    switch (epi) {
    case EPI_ADAMW: return launch_rule<EPI_ADAMW>(a, n, mk, st);
    case EPI_SGD: return launch_rule<EPI_SGD>(a, n, mk, st);
    case EPI_SGDM: return launch_rule<EPI_SGDM>(a, n, mk, st);
    case EPI_ADAGRAD: return launch_rule<EPI_ADAGRAD>(a, n, mk, st);
    case EPI_RMSPROP: return launch_rule<EPI_RMSPROP>(a, n, mk, st);
    case EPI_LION: return launch_rule<EPI_LION>(a, n, mk, st);
    case EPI_NADAM: return launch_rule<EPI_NADAM>(a, n, mk, st);
    case EPI_RADAM: return launch_rule<EPI_RADAM>(a, n, mk, st);
    case EPI_ADAMAX: return launch_rule<EPI_ADAMAX>(a, n, mk, st);
    case EPI_MUON: return launch_rule<EPI_MUON>(a, n, mk, st);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_fused_wfp8(const Args *a, int n, int mk, hipStream_t st)
{
    if (mk == MK_FP8) return launch_group<BP_F, BQ_F, MK_FP8, EPI_ADAMW_WFP8>(a, n, st);
    if (mk == MK_BF16) return launch_group<BP_F, BQ_F, MK_BF16, EPI_ADAMW_WFP8>(a, n, st);
    return hipErrorInvalidValue;
}

hipError_t launch_fused(const Args &a, int mk, hipStream_t st)
{
    return launch_fused_group(&a, 1, mk, st);
}

hipError_t launch_wgrad(const Args &a, int grad_f32, hipStream_t st)
{
    if (grad_f32) return launch_group<BP_F, BQ_F, MK_BF16, EPI_STORE_F32>(&a, 1, st);
    return launch_group<BP_F, BQ_F, MK_BF16, EPI_STORE_BF16>(&a, 1, st);
}

hipError_t launch_adamw(const Args &a0, int mk, int grad_f32, hipStream_t st)
{
    int n;
    if (mk == MK_I8) {
        Args a = with_grid(a0, BP_I8, BQ_I8, n);
        if (grad_f32)
            hipLaunchKernelGGL((adamw_kernel<BP_I8, BQ_I8, MK_I8, true>), dim3(n), dim3(NROLE), 0, st, a);
        else
            hipLaunchKernelGGL((adamw_kernel<BP_I8, BQ_I8, MK_I8, false>), dim3(n), dim3(NROLE), 0, st, a);
    } else if (mk == MK_I8R64) {
        Args a = with_grid(a0, BP_F, BQ_F, n);
        if (grad_f32)
            hipLaunchKernelGGL((adamw_kernel<BP_F, BQ_F, MK_I8R64, true>), dim3(n), dim3(NROLE), 0, st, a);
        else
            hipLaunchKernelGGL((adamw_kernel<BP_F, BQ_F, MK_I8R64, false>), dim3(n), dim3(NROLE), 0, st, a);
    } else if (mk == MK_BF16) {
        Args a = with_grid(a0, BP_F, BQ_F, n);
        if (grad_f32)
            hipLaunchKernelGGL((adamw_kernel<BP_F, BQ_F, MK_BF16, true>), dim3(n), dim3(NROLE), 0, st, a);
        else
            hipLaunchKernelGGL((adamw_kernel<BP_F, BQ_F, MK_BF16, false>), dim3(n), dim3(NROLE), 0, st, a);
    } else {
        Args a = with_grid(a0, BP_F, BQ_F, n);
        if (grad_f32)
            hipLaunchKernelGGL((adamw_kernel<BP_F, BQ_F, MK_F32, true>), dim3(n), dim3(NROLE), 0, st, a);
        else
            hipLaunchKernelGGL((adamw_kernel<BP_F, BQ_F, MK_F32, false>), dim3(n), dim3(NROLE), 0, st, a);
    }
    return hipGetLastError();
}

}  // namespace forge_impl
