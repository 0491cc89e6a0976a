// forge_dx.hip -- gfx950 (CDNA4) kernel for the layer's input gradient dX = dY W.
//
// The fused step overwrites W in place, so the chain rule's input gradient must be formed
// from the weight as it was before the update (Sec. 2.2, the paragraph after Eq. tile;
// Algorithm 1, first line; the ordering remark of App. A): the layer-level backward runs
// this GEMM first and the fused step after it, in stream order.
//
// dX [T, d_in] = sum over segments s of dY_s [T, d_out_s] W_s [d_out_s, d_in].  With one
// segment this is dY W.  Projections that read the same input (q, k and v; an MLP's gate
// and up) each contribute a term to that input's gradient; one launch sums them by running
// the GEMM's K loop over their concatenated d_out axes, with one rounding to bf16 at the end.
//
// One workgroup owns an output tile dX[t0 : t0+BT, q0 : q0+BQ] held in fp32 registers: four
// waves for 64- and 128-row tiles of 128 columns, eight waves (two per SIMD, each holding
// 128 x 64 outputs) for 256 x 256 tiles, which halve the LDS fragment reads per flop and
// are chosen once they alone fill the compute units.  MFMA (v_mfma_f32_32x32x16_bf16) operand A is W^T (M = q along d_in, K = p
// along d_out), operand B is dY^T (K = p, N = t); each lane of a 32x32 result holds four
// consecutive q of one token row, which is the order the tile is staged in for its stores.
#include "forge_device.h"

namespace forge_impl {

#ifndef FORGE_DX_BT               // token rows per tile: 64, 128, 256, or 0 to choose by shape
#define FORGE_DX_BT 0
#endif

constexpr int DX_NS = 4;          // LDS ring depth (chunks)

constexpr int DX_NT = 256;        // threads per workgroup of the 64- and 128-row tiles
constexpr int DX_BQ = 128;        // their columns of dX per tile

// Operand path: a ring of NS LDS stages; a stage holds one chunk of BK rows p of W
// (columns q0 .. q0+BQ-1, row pitch 2*BQ bytes) followed by the matching BK columns of dY
// for the tile's BT token rows (2*BK-byte rows).  Chunks are copied HBM/L2 -> LDS by buffer
// loads that write LDS directly (NS-1 chunks in flight).  Each chunk gets buffers of
// its own: W's ends at the segment's last row, so rows past d_out read zero; dY's starts
// at the chunk's first column of the tile's first row, and a piece past the segment's
// d_out or past row T gets OOR_OFFSET, which reads zero.  (Zero, not the next row's
// values: a finite weight times an Inf there would otherwise leak a NaN into dX.)
//
// Fragments: W's (8 consecutive p of one q) come from the transposing LDS read
// ds_read_b64_tr_b16 -- lane s of each 16 points at row p0 + s/4, column c0 + 4 (s%4), so
// that lane i receives column c0 + i, rows p0 .. p0+3; dY's (8 consecutive p of one t) are
// one 16-byte ds_read_b128 each.
template <int BT, int BQ, int NA, int NB, int BK, int NS, int NW = 4>
struct DxTile {
    static_assert(BK == 32 || BK == 64, "chunks of 32 or 64 rows of W");
    static constexpr int WQ = BQ / (32 * NA);            // waves along q (each 32*NA columns)
    static constexpr int WT = BT / (32 * NB);            // waves along t (each 32*NB rows)
    static_assert(WQ * WT == NW, "waves");
    static constexpr int WROWB = BQ * 2;                 // LDS bytes per W row
    static constexpr int YROWB = BK * 2;                 // LDS bytes per dY row
    static constexpr int PPR = BK / 8;                   // 16-byte pieces per dY row
    static constexpr int KSTEPS = BK / 16;               // MFMA K steps per chunk
    static_assert(WROWB >= 256, "the W swizzle assumes rows of at least 256 bytes");
    static constexpr int WCH = BK * BQ / 8;              // 16-byte pieces of W per chunk
    static constexpr int YCH = BT * BK / 8;              // 16-byte pieces of dY per chunk
    static_assert(WCH % (64 * NW) == 0 && YCH % (64 * NW) == 0, "a wave's k-th DMA is all W or all dY");
    static constexpr int KW = WCH / (64 * NW);           // DMA instructions per wave for W
    static constexpr int DPC = (WCH + YCH) / (64 * NW);  // DMA instructions per wave per chunk
    static constexpr int KY = DPC - KW;
    static constexpr int STAGE_BYTES = (WCH + YCH) * 16;
    static constexpr int OP = BQ + 4;                    // fp32 pitch of the staged output tile
    static constexpr int OPB = BQ + 8;                   // bf16 pitch of the staged output tile
    static constexpr bool OUT_BF16 = BT * OP * 4 > 96 * 1024;   // big tiles stage rounded bf16
    static constexpr int OUT_BYTES = OUT_BF16 ? BT * OPB * 2 : BT * OP * 4;
    static constexpr int RING = NS * STAGE_BYTES;
    static constexpr int LDS_BYTES = RING > OUT_BYTES ? RING : OUT_BYTES;
    static constexpr int NRD = 2 * NA + NB;              // LDS reads per 16-row K step

    f32x16_t acc[NA][NB];
    uint32_t wo[KW];           // W pieces: byte offsets in a chunk's W buffer (fixed per tile)
    int yr[KY];                // dY pieces: token row in the tile, -1 past T
    int yc[KY];                // dY pieces: column within the chunk (multiple of 8)
    uint32_t ta[NA];           // LDS offsets of this lane's W fragment rows
    uint32_t tb[NB][KSTEPS];   // LDS offsets of this lane's dY fragments, per 16-row K step

    // W rows: half a wave's transposing read covers 4 rows x 4 aligned pieces (64 B per
    // row); XOR-ing the piece index with 4*(p%4) gives each row its own quarter of the 64
    // banks.  dY rows: sixteen lanes of a 16-byte read cover 16 consecutive rows at one
    // piece index; XOR-ing it with (t/4)%4 (64-byte rows) or (t/2)%8 (128-byte rows)
    // spreads them over all 64 banks.
    static __device__ __forceinline__ int wswz(int p) { return 4 * (p & 3); }
    static __device__ __forceinline__ int yswz(int t) { return BK == 32 ? (t >> 2) & 3 : (t >> 1) & 7; }

    __device__ __forceinline__ void setup(const DxArgs &g, int t0, int q0, int wave, int lane)
    {
#pragma unroll
        for (int k = 0; k < KW; ++k) {
            const int L = (k * NW + wave) * 64 + lane;
            const int r = L / (BQ / 8);
            const int col = q0 + 8 * ((L % (BQ / 8)) ^ wswz(r));
            const uint64_t off = ((uint64_t)r * (uint64_t)g.d_in + (uint64_t)col) * 2u;
            wo[k] = (col < g.d_in && off < OOR_OFFSET) ? (uint32_t)off : OOR_OFFSET;
        }
#pragma unroll
        for (int k = 0; k < KY; ++k) {
            const int L = (k * NW + wave) * 64 + lane;
            const int t = L / PPR;
            yr[k] = (t0 + t < g.T) ? t : -1;
            yc[k] = 8 * ((L % PPR) ^ yswz(t));
        }
        const int wq = wave % WQ, wt = wave / WQ;
        const int s = lane & 15;
        const int prow = 8 * (lane >> 5) + (s >> 2);
        const int half = (s & 1) * 8;
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            const int qb = wq * 32 * NA + i * 32 + 16 * ((lane >> 4) & 1);
            const int cq = (qb / 8 + ((s & 3) >> 1)) ^ wswz(prow);
            ta[i] = prow * WROWB + cq * 16 + half;
        }
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int t = wt * 32 * NB + j * 32 + (lane & 31);
#pragma unroll
            for (int ks = 0; ks < KSTEPS; ++ks)
                tb[j][ks] = WCH * 16 + t * YROWB + (((2 * ks + (lane >> 5)) ^ yswz(t)) * 16);
        }
    }

    // DMA of the chunk at rows p0 .. p0+BK-1 of segment sg into a stage.
    __device__ __forceinline__ void issue(const DxArgs &g, const DxSeg &sg, int p0, int t0,
                                          unsigned char *stage, int wave)
    {
        const int rows = min(BK, sg.d_out - p0);
        const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t *>(sg.W + (size_t)p0 * (size_t)g.d_in), (short)0,
            (int)((uint32_t)rows * (uint32_t)g.d_in * 2u), 0x00020000);
        const __amdgpu_buffer_rsrc_t ry = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t *>(sg.dY + (size_t)t0 * (size_t)sg.d_out + p0), (short)0,
            (int)(((uint32_t)(g.T - t0) * (uint32_t)sg.d_out - (uint32_t)p0) * 2u), 0x00020000);
        const int rem = sg.d_out - p0;
#pragma unroll
        for (int k = 0; k < KW; ++k) {
            auto *dst = (__attribute__((address_space(3))) void *)(stage + (k * NW + wave) * 1024);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, dst, 16, wo[k], 0, 0, 0);
        }
#pragma unroll
        for (int k = 0; k < KY; ++k) {
            auto *dst = (__attribute__((address_space(3))) void *)(stage + ((KW + k) * NW + wave) * 1024);
            const uint32_t off = (yr[k] >= 0 && yc[k] < rem)
                                     ? ((uint32_t)yr[k] * (uint32_t)sg.d_out + (uint32_t)yc[k]) * 2u
                                     : OOR_OFFSET;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ry, dst, 16, off, 0, 0, 0);
        }
    }

    template <int OFF>
    static __device__ __forceinline__ void tr_read(v4i16_t &r, uint32_t addr)
    {
        asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF) : "memory");
    }
    static __device__ __forceinline__ void read128(bf16x8_t &r, uint32_t addr)
    {
        asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(addr) : "memory");
    }
    static __device__ __forceinline__ bf16x8_t cat(v4i16_t lo, v4i16_t hi)
    {
        return __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }

    // 32 rows of a chunk (half h of a 64-row chunk): two 16-row K steps.  All reads are
    // issued up front; the first step's MFMAs wait only for its own reads (LDS returns in
    // order).
    template <int H>
    __device__ __forceinline__ void compute(uint32_t st)
    {
        constexpr int R = 32 * H * WROWB;                 // W rows of this half
        v4i16_t fa[2][NA][2];
        bf16x8_t fb[2][NB];
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            tr_read<R + 0 * WROWB>(fa[0][i][0], st + ta[i]);
            tr_read<R + 4 * WROWB>(fa[0][i][1], st + ta[i]);
        }
#pragma unroll
        for (int j = 0; j < NB; ++j) read128(fb[0][j], st + tb[j][2 * H]);
        // at most 15 LDS reads outstanding (lgkmcnt's range): with many fragments per
        // step the second step's reads follow the first step's wait
        constexpr bool ALL_AHEAD = 2 * NRD <= 15;
        static_assert(NRD <= 15, "lgkmcnt range");
        if constexpr (!ALL_AHEAD) wait_lgkm<0>(fa[0], fb[0]);
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            tr_read<R + 16 * WROWB>(fa[1][i][0], st + ta[i]);
            tr_read<R + 20 * WROWB>(fa[1][i][1], st + ta[i]);
        }
#pragma unroll
        for (int j = 0; j < NB; ++j) read128(fb[1][j], st + tb[j][2 * H + 1]);
        if constexpr (ALL_AHEAD) wait_lgkm<NRD>(fa[0], fb[0]);
#pragma unroll
        for (int i = 0; i < NA; ++i)
#pragma unroll
            for (int j = 0; j < NB; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cat(fa[0][i][0], fa[0][i][1]), fb[0][j],
                                                                     acc[i][j], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);   // keep the first step's MFMAs ahead of the next wait
        wait_lgkm<0>(fa[1], fb[1]);
#pragma unroll
        for (int i = 0; i < NA; ++i)
#pragma unroll
            for (int j = 0; j < NB; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cat(fa[1][i][0], fa[1][i][1]), fb[1][j],
                                                                     acc[i][j], 0, 0, 0);
    }

    // Wait until at most N LDS reads of this wave are outstanding; the fragments named
    // are the ones that wait guarantees (so the compiler keeps their uses after it).
    template <int N>
    static __device__ __forceinline__ void wait_lgkm(v4i16_t (&fa)[NA][2], bf16x8_t (&fb)[NB])
    {
        asm volatile("s_waitcnt lgkmcnt(%0)" ::"i"(N) : "memory");
#pragma unroll
        for (int i = 0; i < NA; ++i) asm volatile("" : "+v"(fa[i][0]), "+v"(fa[i][1]));
#pragma unroll
        for (int j = 0; j < NB; ++j) asm volatile("" : "+v"(fb[j]));
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
            if (younger >= Y)
                asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"i"(DPC * Y) : "memory");
            else
                wait_chunk<Y - 1>(younger);
        }
    }

    // The K loop over every chunk of every segment.  Chunks never straddle segments; the
    // issue cursor (segment si, row p0) runs NS-1 chunks ahead of the compute.
    __device__ __forceinline__ void run(const DxArgs &g, int t0, int q0, unsigned char *lds, int wave,
                                        int lane)
    {
#pragma unroll
        for (int i = 0; i < NA; ++i)
#pragma unroll
            for (int j = 0; j < NB; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
        setup(g, t0, q0, wave, lane);
        // Issue cursor: segment si (its descriptor kept in registers), row p0.
        int si = 0, p0 = 0;
        DxSeg sg = g.s[0];
        auto advance = [&]() {
            p0 += BK;
            if (p0 >= sg.d_out) {
                ++si;
                p0 = 0;
                if (si < g.n) sg = g.s[si];
            }
        };
        const int nch = g.nch;
#pragma unroll
        for (int c = 0; c < NS - 1; ++c)
            if (c < nch) {
                issue(g, sg, p0, t0, lds + c * STAGE_BYTES, wave);
                advance();
            }
        const uint32_t base = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)lds;
        for (int c = 0; c < nch; ++c) {
            wait_chunk(min(NS - 2, nch - 1 - c));
            const uint32_t st = base + (uint32_t)((c % NS) * STAGE_BYTES);
            compute<0>(st);
            if constexpr (BK == 64) compute<1>(st);
            if (c + NS - 1 < nch) {
                issue(g, sg, p0, t0, lds + ((c + NS - 1) % NS) * STAGE_BYTES, wave);
                advance();
            }
        }
        lds_barrier();   // every wave is done reading the ring, which the output reuses
    }

    // Accumulators -> LDS as dX[t][q] (fp32), then coalesced bf16 stores (round to
    // nearest even): 16 lanes cover one 128-column row with 16-byte stores.
    __device__ __forceinline__ void store(const DxArgs &g, int t0, int q0, unsigned char *lds, int wave,
                                          int lane, int tid) const
    {
        if constexpr (OUT_BF16) {
            store_bf16(g, t0, q0, lds, wave, lane, tid);
            return;
        }
        float *Os = reinterpret_cast<float *>(lds);
        const int wq = wave % WQ, wt = wave / WQ;
#pragma unroll
        for (int i = 0; i < NA; ++i)
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                const int t = wt * 32 * NB + j * 32 + (lane & 31);
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const int q = wq * 32 * NA + i * 32 + q4 * 8 + (lane >> 5) * 4;
                    const f32x4_t v = {acc[i][j][4 * q4], acc[i][j][4 * q4 + 1], acc[i][j][4 * q4 + 2],
                                       acc[i][j][4 * q4 + 3]};
                    *reinterpret_cast<f32x4_t *>(Os + t * OP + q) = v;
                }
            }
        lds_barrier();
        constexpr int LPR = BQ / 8, RPP = 64 * NW / LPR;
        const int rs = tid / LPR, qo = (tid % LPR) * 8, q = q0 + qo;
        if (q >= g.d_in) return;
#pragma unroll
        for (int r = 0; r < BT; r += RPP) {
            const int t = r + rs;
            if (t0 + t >= g.T) break;
            const float *o = Os + t * OP + qo;
            const f32x4_t a = *reinterpret_cast<const f32x4_t *>(o);
            const f32x4_t b = *reinterpret_cast<const f32x4_t *>(o + 4);
            const u32x4_t w = {pack_bf16(a[0], a[1]), pack_bf16(a[2], a[3]), pack_bf16(b[0], b[1]),
                               pack_bf16(b[2], b[3])};
            *reinterpret_cast<u32x4_t *>(g.dX + (size_t)(t0 + t) * (size_t)g.d_in + q) = w;
        }
    }

    // Big tiles: each accumulator rounded to bf16 (round to nearest even) in registers, the
    // tile staged as bf16, then 16-byte stores of whole rows.  Rounding before or after the
    // staging gives the same bits.
    __device__ __forceinline__ void store_bf16(const DxArgs &g, int t0, int q0, unsigned char *lds, int wave,
                                               int lane, int tid) const
    {
        uint16_t *Ob = reinterpret_cast<uint16_t *>(lds);
        const int wq = wave % WQ, wt = wave / WQ;
#pragma unroll
        for (int i = 0; i < NA; ++i)
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                const int t = wt * 32 * NB + j * 32 + (lane & 31);
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const int q = wq * 32 * NA + i * 32 + q4 * 8 + (lane >> 5) * 4;
                    const u32x2_t v = {pack_bf16(acc[i][j][4 * q4], acc[i][j][4 * q4 + 1]),
                                       pack_bf16(acc[i][j][4 * q4 + 2], acc[i][j][4 * q4 + 3])};
                    *reinterpret_cast<u32x2_t *>(Ob + t * OPB + q) = v;
                }
            }
        lds_barrier();
        constexpr int LPR = BQ / 8, RPP = 64 * NW / LPR;
        const int rs = tid / LPR, qo = (tid % LPR) * 8, q = q0 + qo;
        if (q >= g.d_in) return;
#pragma unroll
        for (int r = 0; r < BT; r += RPP) {
            const int t = r + rs;
            if (t0 + t >= g.T) break;
            const u32x4_t w = *reinterpret_cast<const u32x4_t *>(Ob + t * OPB + qo);
            *reinterpret_cast<u32x4_t *>(g.dX + (size_t)(t0 + t) * (size_t)g.d_in + q) = w;
        }
    }
};

// 128-row tiles use 32-row chunks (66 KB of LDS: two workgroups per CU); 64-row tiles,
// which run one workgroup per CU on the short token axes they are chosen for, use 64-row
// chunks (96 KB), which halves the barriers per K and keeps twice the bytes in flight.
// 256 x 256 tiles: eight waves, 32-row chunks (128 KB ring), output staged as bf16 (132 KB),
// one workgroup per CU.
template <int BT, int NA, int NB, int BK, int NS, int BQ = DX_BQ, int NW = 4>
__global__ void __launch_bounds__(64 * NW, (BK == 64 || NW > 4) ? 1 : 2) dx_kernel(DxArgs g)
{
    using L = DxTile<BT, BQ, NA, NB, BK, NS, NW>;
    __shared__ __attribute__((aligned(16))) unsigned char smem[L::LDS_BYTES];
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    int tt, tq;
    tile_of(blockIdx.x, gridDim.x, g.tiles_t, g.tiles_q, g.group_t, tt, tq);
    const int t0 = tt * BT, q0 = tq * BQ;
    L tile;
    tile.run(g, t0, q0, smem, wave, lane);
    tile.store(g, t0, q0, smem, wave, lane, tid);
}

// Token rows per tile: 256 (256 x 256 tiles, 2x4 waves of 128x64) once those alone cover
// every compute unit; else 128 (2x2 waves of 64x64) once the 128x128 tiles do; else 64 (4x1
// waves of 32 columns x 64 rows), which doubles the tile count for the short token axes of
// fine-tuning-sized batches.  Every choice sums over K in the same order: dX is the same
// bits whichever tile computes it.
static int dx_rows(int T, int d_in)
{
    if (FORGE_DX_BT) return FORGE_DX_BT;
    if ((long)((T + 255) / 256) * (long)((d_in + 255) / 256) >= (long)device_cu_count()) return 256;
    const long t128 = (long)((T + 127) / 128) * (long)((d_in + DX_BQ - 1) / DX_BQ);
    return t128 >= (long)device_cu_count() ? 128 : 64;
}

hipError_t launch_dx(const DxSeg *s, int n, uint16_t *dX, int T, int d_in, hipStream_t st)
{
    if (T == 0 || d_in == 0) return hipSuccess;
    DxArgs g;
    g.n = n;
    g.nch = 0;
    for (int i = 0; i < MAX_GROUP; ++i) g.s[i] = i < n ? s[i] : DxSeg{nullptr, nullptr, 0};
    const int bt = dx_rows(T, d_in);
    const int bk = bt == 64 ? 64 : 32;
    for (int i = 0; i < n; ++i) g.nch += (s[i].d_out + bk - 1) / bk;
    g.dX = dX;
    g.T = T;
    g.d_in = d_in;
    const int bq = bt == 256 ? 256 : DX_BQ;
    g.tiles_t = (T + bt - 1) / bt;
    g.tiles_q = (d_in + bq - 1) / bq;
    g.group_t = g.tiles_t < 16 ? g.tiles_t : 16;
    const int ntiles = g.tiles_t * g.tiles_q;
    if (bt == 256)
        hipLaunchKernelGGL((dx_kernel<256, 4, 2, 32, DX_NS, 256, 8>), dim3(ntiles), dim3(512), 0, st, g);
    else if (bt == 128)
        hipLaunchKernelGGL((dx_kernel<128, 2, 2, 32, DX_NS>), dim3(ntiles), dim3(DX_NT), 0, st, g);
    else
        hipLaunchKernelGGL((dx_kernel<64, 1, 2, 64, DX_NS>), dim3(ntiles), dim3(DX_NT), 0, st, g);
    return hipGetLastError();
}

}  // namespace forge_impl
