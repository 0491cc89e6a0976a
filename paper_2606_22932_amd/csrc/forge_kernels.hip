// forge_kernels.hip -- gfx950 (CDNA4) kernels for the fused weight-gradient + AdamW step.
//
// One workgroup owns one tile of W (FORGE Sec. 2.2, Eq. tile, Algorithm 1) and has two
// roles of four waves each:
//
//   math waves   stage X and dY token chunks from HBM/L2 into LDS (transposing them so
//                that the token axis, the GEMM's K, is contiguous), and accumulate
//                G_tile = dY_tile^T X_tile with v_mfma_f32_32x32x16_bf16 into fp32
//                registers; at the end they drop the accumulator tile into LDS.
//   stream waves issue every global load of the tile's W, m, v (and int8 scales) when
//                the workgroup starts, so that this HBM traffic overlaps the mainloop
//                (vmcnt is per wave, so the math waves never wait on it); then they run
//                the AdamW epilogue on the LDS copy of G with coalesced 16-byte accesses
//                and store W, m, v.  G never leaves the chip.
//
// The two-kernel comparison path reuses the same pieces: the store-G GEMM runs the same
// mainloop with an epilogue that writes G, and the stand-alone optimizer stages a tile
// of a materialised G into LDS and runs the same epilogue code.
#include "forge_internal.h"

namespace forge_impl {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int TK = 32;          // tokens per pipeline chunk (the GEMM's K step)
constexpr int OPP = TK + 8;     // LDS operand row pitch in bf16 (80 B: conflict-free b128 reads)
constexpr int NROLE = 256;      // threads per role (4 waves)
constexpr int NT = 2 * NROLE;   // threads per fused workgroup
constexpr int I8_BLOCK = 256;   // rows of d_out sharing one int8 scale

// Tile shapes: (rows along d_out) x (cols along d_in).  int8 tiles are exactly one scale
// block tall so that the block absmax closes inside the workgroup.
constexpr int BP_F = 128, BQ_F = 128;
constexpr int BP_I8 = 256, BQ_I8 = 64;

// ------------------------------------------------------------------------ small helpers

__device__ __forceinline__ void lds_barrier()
{
    // Wait for this wave's LDS traffic only, then barrier: outstanding global loads (the
    // stream waves' prefetch) stay in flight across it.
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    bf16x2_t r = {(__bf16)lo, (__bf16)hi};   // v_cvt_pk_bf16_f32: round to nearest even
    return __builtin_bit_cast(uint32_t, r);
}

template <typename T> __device__ __forceinline__ T ld_nt(const void *p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const T *>(p));
}
template <typename T> __device__ __forceinline__ void st_nt(void *p, T v)
{
    __builtin_nontemporal_store(v, reinterpret_cast<T *>(p));
}

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

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own L2): give
// each XCD a contiguous run of tiles, and walk that run in groups of `group_p` tile rows
// so that concurrently resident tiles share their dY row slabs and X column slabs.
__device__ __forceinline__ void tile_of(int bid, int ntiles, int tiles_p, int tiles_q,
                                        int group_p, int &tp, int &tq)
{
    const int k = ntiles >> 3, r = ntiles & 7;
    const int x = bid & 7, s = bid >> 3;
    const int t = (x < r) ? x * (k + 1) + s : r * (k + 1) + (x - r) * k + s;
    const int per_group = group_p * tiles_q;
    const int g = t / per_group;
    const int first = g * group_p;
    const int gsz = min(group_p, tiles_p - first);
    const int within = t - g * per_group;
    tp = first + within % gsz;
    tq = within / gsz;
}

// ------------------------------------------------------------------------ mainloop

// G^T tile (rows q along d_in, cols p along d_out) = X_tile^T dY_tile, accumulated in
// fp32.  MFMA operand A is X (M = q), operand B is dY (N = p); each lane of a 32x32
// result holds 4 consecutive q for one p, which is the order G is staged in below.
template <int BP, int BQ>
struct Mainloop {
    static constexpr int WQ = BQ / 64;                   // waves along q
    static constexpr int WP = BP / 64;                   // waves along p
    static_assert(WQ * WP == 4, "four math waves, 64x64 each");
    static constexpr int XBLK = (BQ / 8) * (TK / 4);     // 4-token x 8-column blocks of X per chunk
    static constexpr int YBLK = (BP / 8) * (TK / 4);
    static constexpr int NBLK = XBLK + YBLK;
    static constexpr int NPER = (NBLK + NROLE - 1) / NROLE;
    static constexpr int XS_ELEMS = BQ * OPP;            // one stage of X in LDS (bf16)
    static constexpr int STAGE_ELEMS = (BP + BQ) * OPP;
    static constexpr int LDS_BYTES = 2 * STAGE_ELEMS * 2;

    f32x16_t acc[2][2];                                  // [q sub-tile][p sub-tile]
    u32x4_t stg[NPER][4];                                // one chunk's global loads

    __device__ __forceinline__ void gload(const Args &a, int p0, int q0, int c, int tid)
    {
        const int t0 = c * TK;
#pragma unroll
        for (int j = 0; j < NPER; ++j) {
            const int b = tid + j * NROLE;
            if (NBLK % NROLE != 0 && b >= NBLK) break;
            const uint16_t *base;
            int ld, col, lim, tt;
            if (b < XBLK) {
                col = q0 + (b % (BQ / 8)) * 8; tt = (b / (BQ / 8)) * 4;
                base = a.X; ld = a.d_in; lim = a.d_in;
            } else {
                const int b2 = b - XBLK;
                col = p0 + (b2 % (BP / 8)) * 8; tt = (b2 / (BP / 8)) * 4;
                base = a.dY; ld = a.d_out; lim = a.d_out;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int t = t0 + tt + i;
                u32x4_t v = {0u, 0u, 0u, 0u};
                if (t < a.T && col < lim)
                    v = *reinterpret_cast<const u32x4_t *>(base + (size_t)t * ld + col);
                stg[j][i] = v;
            }
        }
    }

    // Transpose each 4-token x 8-column block in registers and write it as eight 4-token
    // rows (one per column), so LDS holds [column][token] with the token axis contiguous.
    __device__ __forceinline__ void lstore(uint16_t *stage, int tid)
    {
#pragma unroll
        for (int j = 0; j < NPER; ++j) {
            const int b = tid + j * NROLE;
            if (NBLK % NROLE != 0 && b >= NBLK) break;
            uint16_t *row;
            if (b < XBLK) {
                row = stage + ((b % (BQ / 8)) * 8) * OPP + (b / (BQ / 8)) * 4;
            } else {
                const int b2 = b - XBLK;
                row = stage + XS_ELEMS + ((b2 % (BP / 8)) * 8) * OPP + (b2 / (BP / 8)) * 4;
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t r0 = stg[j][0][k], r1 = stg[j][1][k];
                const uint32_t r2 = stg[j][2][k], r3 = stg[j][3][k];
                u32x2_t even = {(r0 & 0xFFFFu) | (r1 << 16), (r2 & 0xFFFFu) | (r3 << 16)};
                u32x2_t odd = {(r0 >> 16) | (r1 & 0xFFFF0000u), (r2 >> 16) | (r3 & 0xFFFF0000u)};
                *reinterpret_cast<u32x2_t *>(row + (2 * k) * OPP) = even;
                *reinterpret_cast<u32x2_t *>(row + (2 * k + 1) * OPP) = odd;
            }
        }
    }

    __device__ __forceinline__ void compute(const uint16_t *stage, int wave, int lane)
    {
        const int wq = wave % WQ, wp = wave / WQ;
        const uint16_t *xs = stage + (wq * 64 + (lane & 31)) * OPP + (lane >> 5) * 8;
        const uint16_t *ys = stage + XS_ELEMS + (wp * 64 + (lane & 31)) * OPP + (lane >> 5) * 8;
#pragma unroll
        for (int ks = 0; ks < TK / 16; ++ks) {
            bf16x8_t A[2], B[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                A[i] = *reinterpret_cast<const bf16x8_t *>(xs + i * 32 * OPP + ks * 16);
                B[i] = *reinterpret_cast<const bf16x8_t *>(ys + i * 32 * OPP + ks * 16);
            }
#pragma unroll
            for (int iq = 0; iq < 2; ++iq)
#pragma unroll
                for (int ip = 0; ip < 2; ++ip)
                    acc[iq][ip] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A[iq], B[ip],
                                                                          acc[iq][ip], 0, 0, 0);
        }
    }

    // Runs the whole token loop; executes exactly nbar(T) LDS barriers.
    __device__ __forceinline__ void run(const Args &a, int p0, int q0, uint16_t *lds, int tid,
                                        int wave, int lane)
    {
#pragma unroll
        for (int iq = 0; iq < 2; ++iq)
#pragma unroll
            for (int ip = 0; ip < 2; ++ip)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[iq][ip][r] = 0.0f;
        const int nch = (a.T + TK - 1) / TK;
        if (nch == 0) return;
        gload(a, p0, q0, 0, tid);
        lstore(lds, tid);
        lds_barrier();
        for (int c = 0; c < nch; ++c) {
            const bool more = c + 1 < nch;
            if (more) gload(a, p0, q0, c + 1, tid);
            compute(lds + (c & 1) * STAGE_ELEMS, wave, lane);
            if (more) lstore(lds + ((c + 1) & 1) * STAGE_ELEMS, tid);
            lds_barrier();
        }
    }

    static __device__ __forceinline__ int nbar(int T)
    {
        const int nch = (T + TK - 1) / TK;
        return nch > 0 ? nch + 1 : 0;
    }

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
template <int BP, int BQ>
struct EpiMap {
    static constexpr int GP = BQ + 4;           // LDS G row pitch in floats
    static constexpr int LPR = BQ / 8;          // lanes per row
    static constexpr int RPP = NROLE / LPR;     // rows per pass
    static constexpr int NPASS = BP / RPP;
    static constexpr int GS_BYTES = BP * GP * 4;
};

// AdamW on fp32 or bf16 moments.
template <int BP, int BQ, int MK>
struct EpiAdamW {
    using M = EpiMap<BP, BQ>;
    static constexpr bool PREFETCH = (MK == MK_BF16);   // fp32 state would not fit in registers
    u32x4_t pw[PREFETCH ? M::NPASS : 1], pm[PREFETCH ? M::NPASS : 1], pv[PREFETCH ? M::NPASS : 1];

    __device__ __forceinline__ void prefetch(const Args &a, int p0, int q0, int s)
    {
        if constexpr (PREFETCH) {
            const int rs = s / M::LPR, q = q0 + (s % M::LPR) * 8;
#pragma unroll
            for (int i = 0; i < M::NPASS; ++i) {
                const int p = p0 + i * M::RPP + rs;
                pw[i] = pm[i] = pv[i] = u32x4_t{0u, 0u, 0u, 0u};
                if (q < a.d_in && p < a.d_out) {
                    const size_t off = (size_t)p * a.d_in + q;
                    pw[i] = ld_nt<u32x4_t>(a.W + off);
                    pm[i] = ld_nt<u32x4_t>(static_cast<const uint16_t *>(a.m) + off);
                    pv[i] = ld_nt<u32x4_t>(static_cast<const uint16_t *>(a.v) + off);
                }
            }
        }
    }

    __device__ __forceinline__ void run(const Args &a, int p0, int q0, int s, const float *Gs)
    {
        const int rs = s / M::LPR, qo = (s % M::LPR) * 8, q = q0 + qo;
        const Hyper h = a.h;
#pragma unroll
        for (int i = 0; i < M::NPASS; ++i) {
            const int p = p0 + i * M::RPP + rs;
            const bool ok = q < a.d_in && p < a.d_out;
            const size_t off = (size_t)p * a.d_in + q;
            const float *gr = Gs + (i * M::RPP + rs) * M::GP + qo;
            const f32x4_t g0 = *reinterpret_cast<const f32x4_t *>(gr);
            const f32x4_t g1 = *reinterpret_cast<const f32x4_t *>(gr + 4);
            const float g[8] = {g0[0], g0[1], g0[2], g0[3], g1[0], g1[1], g1[2], g1[3]};
            u32x4_t w4;
            float mf[8], vf[8];
            if constexpr (PREFETCH) {
                w4 = pw[i];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    mf[2 * k] = bf_lo(pm[i][k]); mf[2 * k + 1] = bf_hi(pm[i][k]);
                    vf[2 * k] = bf_lo(pv[i][k]); vf[2 * k + 1] = bf_hi(pv[i][k]);
                }
            } else {
                w4 = u32x4_t{0u, 0u, 0u, 0u};
                f32x4_t m0 = {0, 0, 0, 0}, m1 = m0, v0 = m0, v1 = m0;
                if (ok) {
                    w4 = ld_nt<u32x4_t>(a.W + off);
                    const float *mp = static_cast<const float *>(a.m) + off;
                    const float *vp = static_cast<const float *>(a.v) + off;
                    m0 = ld_nt<f32x4_t>(mp); m1 = ld_nt<f32x4_t>(mp + 4);
                    v0 = ld_nt<f32x4_t>(vp); v1 = ld_nt<f32x4_t>(vp + 4);
                }
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    mf[k] = m0[k]; mf[k + 4] = m1[k];
                    vf[k] = v0[k]; vf[k + 4] = v1[k];
                }
            }
            float wo[8], mo[8], vo[8];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                float rv;
                adamw_elem(g[2 * k], bf_lo(w4[k]), mf[2 * k], vf[2 * k], h, wo[2 * k], mo[2 * k],
                           vo[2 * k], rv);
                adamw_elem(g[2 * k + 1], bf_hi(w4[k]), mf[2 * k + 1], vf[2 * k + 1], h,
                           wo[2 * k + 1], mo[2 * k + 1], vo[2 * k + 1], rv);
            }
            if (ok) {
                u32x4_t wn;
#pragma unroll
                for (int k = 0; k < 4; ++k) wn[k] = pack_bf16(wo[2 * k], wo[2 * k + 1]);
                st_nt<u32x4_t>(a.W + off, wn);
                if constexpr (MK == MK_BF16) {
                    u32x4_t mn, vn;
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        mn[k] = pack_bf16(mo[2 * k], mo[2 * k + 1]);
                        vn[k] = pack_bf16(vo[2 * k], vo[2 * k + 1]);
                    }
                    st_nt<u32x4_t>(static_cast<uint16_t *>(a.m) + off, mn);
                    st_nt<u32x4_t>(static_cast<uint16_t *>(a.v) + off, vn);
                } else {
                    float *mp = static_cast<float *>(a.m) + off;
                    float *vp = static_cast<float *>(a.v) + off;
                    st_nt<f32x4_t>(mp, f32x4_t{mo[0], mo[1], mo[2], mo[3]});
                    st_nt<f32x4_t>(mp + 4, f32x4_t{mo[4], mo[5], mo[6], mo[7]});
                    st_nt<f32x4_t>(vp, f32x4_t{vo[0], vo[1], vo[2], vo[3]});
                    st_nt<f32x4_t>(vp + 4, f32x4_t{vo[4], vo[5], vo[6], vo[7]});
                }
            }
        }
    }
};

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

    __device__ __forceinline__ void prefetch(const Args &a, int p0, int q0, int s)
    {
        const int rs = s / M::LPR, q = q0 + (s % M::LPR) * 8;
        const bool qok = q < a.d_in;
#pragma unroll
        for (int i = 0; i < M::NPASS; ++i) {
            const int p = p0 + i * M::RPP + rs;
            pw[i] = u32x4_t{0u, 0u, 0u, 0u};
            pm[i] = pv[i] = u32x2_t{0u, 0u};
            if (qok && p < a.d_out) {
                const size_t off = (size_t)p * a.d_in + q;
                pw[i] = ld_nt<u32x4_t>(a.W + off);
                pm[i] = ld_nt<u32x2_t>(static_cast<const int8_t *>(a.m) + off);
                pv[i] = ld_nt<u32x2_t>(static_cast<const int8_t *>(a.v) + off);
            }
        }
        f32x4_t s0 = {0, 0, 0, 0}, s1 = s0, t0 = s0, t1 = s0;
        if (qok) {
            const size_t so = (size_t)(p0 / I8_BLOCK) * a.d_in + q;
            s0 = ld_nt<f32x4_t>(a.ms + so); s1 = ld_nt<f32x4_t>(a.ms + so + 4);
            t0 = ld_nt<f32x4_t>(a.vs + so); t1 = ld_nt<f32x4_t>(a.vs + so + 4);
        }
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

template <int BP, int BQ, int MK, int EPI>
__global__ void __launch_bounds__(NT, 2) fused_kernel(Args a)
{
    using ML = Mainloop<BP, BQ>;
    using EM = EpiMap<BP, BQ>;
    constexpr int RED = (MK == MK_I8 && EPI == EPI_ADAMW) ? 2 * 4 * BQ * 4 : 0;
    constexpr int MAIN = ML::LDS_BYTES > EM::GS_BYTES ? ML::LDS_BYTES : EM::GS_BYTES;
    __shared__ __attribute__((aligned(16))) unsigned char smem[MAIN + RED];
    float *Gs = reinterpret_cast<float *>(smem);
    float *red = reinterpret_cast<float *>(smem + MAIN);

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    int tp, tq;
    tile_of(blockIdx.x, gridDim.x, a.tiles_p, a.tiles_q, a.group_p, tp, tq);
    const int p0 = tp * BP, q0 = tq * BQ;

    if (wave < 4) {
        ML ml;
        ml.run(a, p0, q0, reinterpret_cast<uint16_t *>(smem), tid, wave, lane);
        // the loop's last barrier has retired every read of the operand stages
        ml.template stage_g<EM::GP>(Gs, wave, lane);
        lds_barrier();
        if constexpr (MK == MK_I8 && EPI == EPI_ADAMW) lds_barrier();
        return;
    }

    const int s = tid - NROLE;
    const int nbar = ML::nbar(a.T);
    if constexpr (EPI == EPI_ADAMW) {
        if constexpr (MK == MK_I8) {
            EpiAdamWI8<BP, BQ> ep;
            ep.prefetch(a, p0, q0, s);
            for (int i = 0; i < nbar; ++i) lds_barrier();
            lds_barrier();
            ep.run(a, p0, q0, s, Gs, red);
        } else {
            EpiAdamW<BP, BQ, MK> ep;
            ep.prefetch(a, p0, q0, s);
            for (int i = 0; i < nbar; ++i) lds_barrier();
            lds_barrier();
            ep.run(a, p0, q0, s, Gs);
        }
    } else {
        for (int i = 0; i < nbar; ++i) lds_barrier();
        lds_barrier();
        epi_store_g<BP, BQ, EPI == EPI_STORE_F32>(a, p0, q0, s, Gs);
    }
}

// Stand-alone optimizer over a materialised gradient: 256 threads per tile; each thread
// prefetches its state, the tile of G is staged into LDS (fp32), then the same epilogue
// as the fused kernel runs.
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
        EpiAdamW<BP, BQ, MK> ep;
        ep.prefetch(a, p0, q0, s);
        stage();
        lds_barrier();
        ep.run(a, p0, q0, s, Gs);
    }
}

// ------------------------------------------------------------------------ launchers

TileShape tile_shape(int mk)
{
    if (mk == MK_I8) return TileShape{BP_I8, BQ_I8, TK};
    return TileShape{BP_F, BQ_F, TK};
}

static Args with_grid(Args a, int bp, int bq, int &ntiles)
{
    a.tiles_p = (a.d_out + bp - 1) / bp;
    a.tiles_q = (a.d_in + bq - 1) / bq;
    a.group_p = 8;
    ntiles = a.tiles_p * a.tiles_q;
    return a;
}

hipError_t launch_fused(const Args &a0, int mk, hipStream_t st)
{
    int n;
    if (mk == MK_I8) {
        Args a = with_grid(a0, BP_I8, BQ_I8, n);
        hipLaunchKernelGGL((fused_kernel<BP_I8, BQ_I8, MK_I8, EPI_ADAMW>), dim3(n), dim3(NT), 0, st, a);
    } else if (mk == MK_BF16) {
        Args a = with_grid(a0, BP_F, BQ_F, n);
        hipLaunchKernelGGL((fused_kernel<BP_F, BQ_F, MK_BF16, EPI_ADAMW>), dim3(n), dim3(NT), 0, st, a);
    } else {
        Args a = with_grid(a0, BP_F, BQ_F, n);
        hipLaunchKernelGGL((fused_kernel<BP_F, BQ_F, MK_F32, EPI_ADAMW>), dim3(n), dim3(NT), 0, st, a);
    }
    return hipGetLastError();
}

hipError_t launch_wgrad(const Args &a0, int grad_f32, hipStream_t st)
{
    int n;
    Args a = with_grid(a0, BP_F, BQ_F, n);
    if (grad_f32)
        hipLaunchKernelGGL((fused_kernel<BP_F, BQ_F, MK_BF16, EPI_STORE_F32>), dim3(n), dim3(NT), 0, st, a);
    else
        hipLaunchKernelGGL((fused_kernel<BP_F, BQ_F, MK_BF16, EPI_STORE_BF16>), dim3(n), dim3(NT), 0, st, a);
    return hipGetLastError();
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
