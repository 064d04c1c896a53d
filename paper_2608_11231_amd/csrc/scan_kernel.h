// Chunkwise scan kernel for one recurrent layer (Gated DeltaNet or Mamba-2),
// used by lkv_gdn_chunk_scan / lkv_ssd_chunk_scan (online prefill) and by
// lkv_block_summary (per-block state from zero and per-block transition).
//
// Work unit = (segment s, value head h, row tile).  A row tile is 16*NW rows
// of the dv x dk state (rows of a state evolve independently: the transition
// acts on the dk side only), so a workgroup of NW waves owns 16*NW state rows
// and each wave owns 16 of them.  Chunks of CH tokens are processed in order;
// the fp32 state never leaves registers between chunks.
//
// Per chunk, with token rows Q, K (CH x dk), V (CH x dv), in-chunk cumulative
// log-gates gc_t and b_t = exp(gc_t) (Sec. 2, alpha = exp(g)), the block map of
// Eq. 5 applied to the chunk gives, for Gated DeltaNet (Eq. 3):
//   L = diag(beta) * strictly-lower(exp(gc_t - gc_i) * K K^T)
//   U = (I + L)^{-1} diag(beta) (V - diag(b) K S^T)            (delta-rule write)
//   O = scale (diag(b) Q S^T + lower(exp(gc_t - gc_i) * Q K^T) U)
//   S <- b_C S + U^T diag(exp(gc_C - gc_t)) K
// and for Mamba-2 (Eq. 2; q = C, k = B, v = x, gc = A_h * cumsum(dt)):
//   O = diag(exp(gc)) C S^T + lower(exp(gc_t - gc_i) * C B^T) diag(dt) X
//   S <- exp(gc_C) S + X^T diag(dt * exp(gc_C - gc_t)) B
//
// Precision: bf16 inputs enter the matrix cores exactly.  fp32 operands of the
// products that feed the state (S, the solve, U) are split into bf16 hi + lo
// parts (16 significant bits), and the products use hi*hi + hi*lo + lo*hi, so
// the fp32 state chain keeps ~1e-5 relative accuracy.  Products that only feed
// the bf16 output use the hi part alone.  With fp32 inputs every operand is
// split.
//
// The triangular solve (I + L)^{-1} is blocked by 16: the four 16x16 diagonal
// blocks are inverted by forward substitution (one lane per column), and the
// off-diagonal coupling is applied by block forward substitution on the
// right-hand side, on the matrix cores, wave-locally.
#pragma once
#include "lkv_device.h"

namespace lkv {

enum { FAM_GDN = 0, FAM_SSD = 1 };

struct ScanArgs {
    const int32_t* cu;
    int32_t n_seq;
    int64_t n_tok;
    const void* q;
    const void* k;
    const void* v;
    const void* g;
    const void* beta;
    const float* A;
    int32_t h_qk, h_v, dv;
    int32_t gate_bf16;  // GDN gates stored as bf16
    float scale;
    const float* S_init;  // scan: [n_seq,h_v,dv,dk] or null
    void* out;            // scan: o / y [n_tok,h_v,dv] or null
    float* S_final;       // scan: final state; summary: B_out (may be null)
    float* M_out;         // summary: GDN M [n_seq,h_v,dk,dk] / SSD Lambda [n_seq,h_v], or null
    int32_t summary;      // 0: scan from S_init with outputs; 1: block summary
    int32_t tiles_b;      // row tiles over dv (state rows)
    int32_t tiles_m;      // row tiles over dk (transition rows), GDN summary only
    int32_t nw;           // waves per workgroup
    int32_t n_units;
};

template <int FAM, int DK, int CH, bool F32IO, int NW>
struct ScanLds {
    // Layout: [K | L | N | gates | per-wave gate prefix | V | Q | P], all token
    // tiles row-major.  The block-summary mode has no outputs and stops before Q,
    // so it needs less LDS and fits more workgroups per CU.
    static constexpr int NTC = CH / 16;
    static constexpr int SK = DK + 8;       // bf16 stride of [tok][dk] rows
    static constexpr int SV = 16 * NW + 8;  // bf16 stride of [tok][dv-tile] rows
    static constexpr int SC = CH + 8;       // bf16 stride of [tok][tok] rows
    static constexpr int SCF = CH + 4;      // f32 stride of [tok][tok] rows
    static constexpr int SN = 20;           // f32 stride of a 16x16 block
    static constexpr int PL = F32IO ? 2 : 1;
    static __host__ __device__ constexpr size_t al(size_t x) { return (x + 15) & ~size_t(15); }
    static __host__ __device__ constexpr size_t k_off() { return 0; }
    static __host__ __device__ constexpr size_t l_off() { return al(k_off() + size_t(PL) * CH * SK * 2); }
    static __host__ __device__ constexpr size_t n_off() {
        return al(l_off() + (FAM == FAM_GDN ? size_t(CH) * SCF * 4 : 0));
    }
    static __host__ __device__ constexpr size_t gr_off() {
        return al(n_off() + (FAM == FAM_GDN ? size_t(NTC) * 16 * SN * 4 : 0));
    }
    static __host__ __device__ constexpr size_t be_off() { return al(gr_off() + CH * 4); }
    static __host__ __device__ constexpr size_t gc_off() { return al(be_off() + CH * 4); }
    static __host__ __device__ constexpr size_t v_off() { return al(gc_off() + NW * 64 * 4); }
    static __host__ __device__ constexpr size_t q_off() { return al(v_off() + size_t(PL) * CH * SV * 2); }
    static __host__ __device__ constexpr size_t p_off() { return al(q_off() + size_t(PL) * CH * SK * 2); }
    static __host__ __device__ constexpr size_t end_off() { return al(p_off() + size_t(PL) * CH * SC * 2); }
    static __host__ __device__ constexpr size_t bytes(bool summary) { return summary ? q_off() : end_off(); }
};

// acc += A(rows of an LDS matrix, 16-slices [kb, ke)) x B(acc-layout tiles)
// A row pointers: ah / al point at the lane's row (plane hi / lo); slice kg
// starts at element 16*kg.  B tiles: bh[kg], bl[kg].
template <bool ALO, bool BLO>
__device__ __forceinline__ f32x4 gemm_lds_reg(const bf16* ah, const bf16* al_, const bf16x4* bh,
                                              const bf16x4* bl, int kb, int ke, int g, f32x4 acc) {
    int kg = kb;
    for (; kg + 1 < ke; kg += 2) {
        const bf16x4 a0 = lds4(ah + 16 * kg + 4 * g), a1 = lds4(ah + 16 * kg + 16 + 4 * g);
        acc = mma32(a0, a1, bh[kg], bh[kg + 1], acc);
        if (BLO) acc = mma32(a0, a1, bl[kg], bl[kg + 1], acc);
        if (ALO) {
            const bf16x4 c0 = lds4(al_ + 16 * kg + 4 * g), c1 = lds4(al_ + 16 * kg + 16 + 4 * g);
            acc = mma32(c0, c1, bh[kg], bh[kg + 1], acc);
        }
    }
    if (kg < ke) {
        const bf16x4 a0 = lds4(ah + 16 * kg + 4 * g);
        if (kg == kb) {  // a single 16-slice: the chain is 16-wide MFMAs only
            acc = mma16(a0, bh[kg], acc);
            if (BLO) acc = mma16(a0, bl[kg], acc);
            if (ALO) acc = mma16(lds4(al_ + 16 * kg + 4 * g), bh[kg], acc);
        } else {         // odd tail after 32-wide MFMAs: pad with zeros, never mix shapes
            const bf16x4 z = zero_bf16x4();
            acc = mma32(a0, z, bh[kg], z, acc);
            if (BLO) acc = mma32(a0, z, bl[kg], z, acc);
            if (ALO) acc = mma32(lds4(al_ + 16 * kg + 4 * g), z, bh[kg], z, acc);
        }
    }
    return acc;
}

// acc += M^T(rows c0..c0+15, 16-slices [kb, ke) of M's rows) x B(acc-layout tiles),
// the A fragments read transposed from a row-major LDS matrix M (planes Mh / Ml).
template <bool ALO, bool BLO>
__device__ __forceinline__ f32x4 gemm_ldstr_reg(const bf16* Mh, const bf16* Ml, int stride, int c0,
                                                const bf16x4* bh, const bf16x4* bl, int kb, int ke, int g,
                                                int c, f32x4 acc) {
    int kg = kb;
    for (; kg + 1 < ke; kg += 2) {
        const bf16x4 a0 = lds4_tr(Mh, stride, 16 * kg, c0, g, c), a1 = lds4_tr(Mh, stride, 16 * kg + 16, c0, g, c);
        acc = mma32(a0, a1, bh[kg], bh[kg + 1], acc);
        if (BLO) acc = mma32(a0, a1, bl[kg], bl[kg + 1], acc);
        if (ALO) {
            const bf16x4 c0v = lds4_tr(Ml, stride, 16 * kg, c0, g, c);
            const bf16x4 c1v = lds4_tr(Ml, stride, 16 * kg + 16, c0, g, c);
            acc = mma32(c0v, c1v, bh[kg], bh[kg + 1], acc);
        }
    }
    if (kg < ke) {
        const bf16x4 a0 = lds4_tr(Mh, stride, 16 * kg, c0, g, c);
        if (kg == kb) {
            acc = mma16(a0, bh[kg], acc);
            if (BLO) acc = mma16(a0, bl[kg], acc);
            if (ALO) acc = mma16(lds4_tr(Ml, stride, 16 * kg, c0, g, c), bh[kg], acc);
        } else {
            const bf16x4 z = zero_bf16x4();
            acc = mma32(a0, z, bh[kg], z, acc);
            if (BLO) acc = mma32(a0, z, bl[kg], z, acc);
            if (ALO) acc = mma32(lds4_tr(Ml, stride, 16 * kg, c0, g, c), z, bh[kg], z, acc);
        }
    }
    return acc;
}

// Same with an fp32 LDS A operand that is split on the fly (optionally negated).
template <bool NEG>
__device__ __forceinline__ f32x4 gemm_ldsf_reg(const float* a, const bf16x4* bh, const bf16x4* bl,
                                               int kb, int ke, int g, f32x4 acc) {
    int kg = kb;
    for (; kg + 1 < ke; kg += 2) {
        f32x4 x0 = lds4f(a + 16 * kg + 4 * g), x1 = lds4f(a + 16 * kg + 16 + 4 * g);
        if (NEG) { x0 = -x0; x1 = -x1; }
        const Split4 s0 = split4(x0), s1 = split4(x1);
        acc = mma32(s0.hi, s1.hi, bh[kg], bh[kg + 1], acc);
        acc = mma32(s0.hi, s1.hi, bl[kg], bl[kg + 1], acc);
        acc = mma32(s0.lo, s1.lo, bh[kg], bh[kg + 1], acc);
    }
    if (kg < ke) {
        f32x4 x0 = lds4f(a + 16 * kg + 4 * g);
        if (NEG) x0 = -x0;
        const Split4 s0 = split4(x0);
        if (kg == kb) {
            acc = mma16(s0.hi, bh[kg], acc);
            acc = mma16(s0.hi, bl[kg], acc);
            acc = mma16(s0.lo, bh[kg], acc);
        } else {
            const bf16x4 z = zero_bf16x4();
            acc = mma32(s0.hi, z, bh[kg], z, acc);
            acc = mma32(s0.hi, z, bl[kg], z, acc);
            acc = mma32(s0.lo, z, bh[kg], z, acc);
        }
    }
    return acc;
}

// acc += A(LDS rows) x B(LDS rows)^T over DK, both read with the same pattern.
template <int DK, bool LO>
__device__ __forceinline__ f32x4 gemm_lds_lds(const bf16* ah, const bf16* al_, const bf16* bh,
                                              const bf16* bl, int g, f32x4 acc) {
    constexpr int NK = DK / 16;
#pragma unroll
    for (int kg = 0; kg + 1 < NK; kg += 2) {
        const int o0 = 16 * kg + 4 * g, o1 = o0 + 16;
        const bf16x4 a0 = lds4(ah + o0), a1 = lds4(ah + o1), b0 = lds4(bh + o0), b1 = lds4(bh + o1);
        acc = mma32(a0, a1, b0, b1, acc);
        if (LO) {
            acc = mma32(a0, a1, lds4(bl + o0), lds4(bl + o1), acc);
            acc = mma32(lds4(al_ + o0), lds4(al_ + o1), b0, b1, acc);
        }
    }
    if (NK & 1) {
        const int o0 = 16 * (NK - 1) + 4 * g;
        const bf16x4 a0 = lds4(ah + o0), b0 = lds4(bh + o0);
        acc = mma16(a0, b0, acc);
        if (LO) {
            acc = mma16(a0, lds4(bl + o0), acc);
            acc = mma16(lds4(al_ + o0), b0, acc);
        }
    }
    return acc;
}

__device__ __forceinline__ float load_gate(const void* p, int64_t idx, bool is_bf16) {
    return is_bf16 ? (float)reinterpret_cast<const bf16*>(p)[idx]
                   : reinterpret_cast<const float*>(p)[idx];
}

// A [CH x NCOL] token-major tile of a global tensor, prefetched into registers
// (16-byte vectors, spread over the NTH threads of the workgroup) and later
// committed to LDS as a row-major copy and/or a transposed copy.  Rows t >= n
// read as zero.  The prefetch of chunk c+1 is issued right after chunk c is
// committed, so its latency overlaps chunk c's arithmetic.
template <int CH, int NCOL, bool F32IO, int NTH>
struct TileRegs {
    static constexpr int EPV = F32IO ? 4 : 8;           // elements per 16-byte vector
    static constexpr int VPR = NCOL / EPV;               // vectors per row
    static constexpr int NV = CH * VPR;                  // vectors per tile
    static constexpr int PER = (NV + NTH - 1) / NTH;     // vectors per thread
    uint4 r[PER];

    // element (t, c) of the source lives at base + t*row_stride + c (elements)
    __device__ __forceinline__ void load(const void* base, int64_t row_stride, int n, int tid) {
        constexpr int ES = F32IO ? 4 : 2;
        const char* b = reinterpret_cast<const char*>(base);
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * NTH;
            const int t = idx / VPR, c = (idx % VPR) * EPV;
            uint4 x = uint4{0u, 0u, 0u, 0u};
            if (idx < NV && t < n) x = *reinterpret_cast<const uint4*>(b + (t * row_stride + c) * ES);
            r[i] = x;
        }
    }
    // dst (stride ds, plane offset pofs) and/or dstT[c][t] (stride dts, plane offset pofsT)
    __device__ __forceinline__ void commit(bf16* dst, int ds, int pofs, bf16* dstT, int dts, int pofsT,
                                           int tid) const {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * NTH;
            if (idx >= NV) continue;
            const int t = idx / VPR, c = (idx % VPR) * EPV;
            if (!F32IO) {
                const bf16x8 x = __builtin_bit_cast(bf16x8, r[i]);
                if (dst) *reinterpret_cast<bf16x8*>(dst + t * ds + c) = x;
                if (dstT) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) dstT[(c + e) * dts + t] = x[e];
                }
            } else {
                const Split4 sp = split4(__builtin_bit_cast(f32x4, r[i]));
                if (dst) {
                    *reinterpret_cast<bf16x4*>(dst + t * ds + c) = sp.hi;
                    *reinterpret_cast<bf16x4*>(dst + pofs + t * ds + c) = sp.lo;
                }
                if (dstT) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        dstT[(c + e) * dts + t] = sp.hi[e];
                        dstT[pofsT + (c + e) * dts + t] = sp.lo[e];
                    }
                }
            }
        }
    }
};

template <int FAM, int DK, int CH, bool F32IO, int NW, bool SUMMARY>
__global__ __launch_bounds__(64 * NW) void scan_kernel(ScanArgs p) {
    using Ly = ScanLds<FAM, DK, CH, F32IO, NW>;
    constexpr int NTC = CH / 16, NTK = DK / 16, NTH = 64 * NW;
    constexpr int SK = Ly::SK, SV = Ly::SV, SC = Ly::SC, SCF = Ly::SCF, SN = Ly::SN;
    extern __shared__ __align__(16) char smem[];
    bf16* sK = reinterpret_cast<bf16*>(smem + Ly::k_off());
    bf16* sQ = reinterpret_cast<bf16*>(smem + Ly::q_off());
    bf16* sP = reinterpret_cast<bf16*>(smem + Ly::p_off());
    float* sL = reinterpret_cast<float*>(smem + Ly::l_off());
    float* sN = reinterpret_cast<float*>(smem + Ly::n_off());
    float* sGr = reinterpret_cast<float*>(smem + Ly::gr_off());
    float* sBe = reinterpret_cast<float*>(smem + Ly::be_off());
    float* sGcAll = reinterpret_cast<float*>(smem + Ly::gc_off());
    bf16* sV = reinterpret_cast<bf16*>(smem + Ly::v_off());
    constexpr int KPL = CH * SK;       // plane offset of sK / sQ
    constexpr int PPL = CH * SC;       // plane offset of sP
    constexpr int VPL = CH * SV;       // plane offset of sV

    const int tid = threadIdx.x;
    const int w = tid >> 6, lane = tid & 63, g = lane >> 4, c16 = lane & 15;
    float* sGc = sGcAll + 64 * w;

    // ---- work unit
    const int tiles = p.tiles_b + p.tiles_m;
    const int u = xcd_unit(blockIdx.x, p.n_units);
    const int tile = u % tiles;
    const int h = (u / tiles) % p.h_v;
    const int s = u / (tiles * p.h_v);
    const bool mtile = tile >= p.tiles_b;
    const int row0 = (mtile ? tile - p.tiles_b : tile) * 16 * NW;
    const int my_row = row0 + 16 * w + c16;
    const int hq = h / (p.h_v / p.h_qk);
    int64_t t0 = p.cu[s], t1 = p.cu[s + 1];
    t0 = t0 < 0 ? 0 : (t0 > p.n_tok ? p.n_tok : t0);
    t1 = t1 < t0 ? t0 : (t1 > p.n_tok ? p.n_tok : t1);
    const bool with_out = !SUMMARY && p.out != nullptr;
    const bool load_v = !mtile;
    const float Ah = (FAM == FAM_SSD) ? p.A[h] : 0.f;

    // ---- initial state (acc layout: tile nt holds S[my_row][16nt + 4g + r])
    f32x4 S[NTK];
#pragma unroll
    for (int nt = 0; nt < NTK; ++nt) {
        if (!SUMMARY && p.S_init) {
            S[nt] = *reinterpret_cast<const f32x4*>(
                p.S_init + ((int64_t(s) * p.h_v + h) * p.dv + my_row) * DK + 16 * nt + 4 * g);
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r) S[nt][r] = (mtile && my_row == 16 * nt + 4 * g + r) ? 1.f : 0.f;
        }
    }
    float lam_sum = 0.f;

    // ---- global -> register prefetch of one chunk
    TileRegs<CH, DK, F32IO, NTH> pk, pq;
    TileRegs<CH, 16 * NW, F32IO, NTH> pv;
    float pg = 0.f, pb = 0.f;
    const int64_t qk_rs = (int64_t)p.h_qk * DK, v_rs = (int64_t)p.h_v * p.dv;
    auto prefetch = [&](int64_t c0) {
        const int n = (int)((t1 - c0) < CH ? (t1 - c0) : CH);
        const int64_t qk_off = (c0 * p.h_qk + hq) * (int64_t)DK;
        const int es = F32IO ? 4 : 2;
        pk.load(reinterpret_cast<const char*>(p.k) + qk_off * es, qk_rs, n, tid);
        if (with_out) pq.load(reinterpret_cast<const char*>(p.q) + qk_off * es, qk_rs, n, tid);
        if (load_v) pv.load(reinterpret_cast<const char*>(p.v) + ((c0 * p.h_v + h) * (int64_t)p.dv + row0) * es,
                            v_rs, n, tid);
        if (tid < CH) {
            const int64_t gi = (c0 + tid) * p.h_v + h;
            if (FAM == FAM_GDN) {
                pg = tid < n ? load_gate(p.g, gi, p.gate_bf16) : 0.f;
                pb = tid < n ? load_gate(p.beta, gi, p.gate_bf16) : 0.f;
            } else {
                const float dt = tid < n ? reinterpret_cast<const float*>(p.g)[gi] : 0.f;
                pg = Ah * dt;
                pb = dt;
            }
        }
    };
    if (t0 < t1) prefetch(t0);

    for (int64_t c0 = t0; c0 < t1; c0 += CH) {
        const int n = (int)((t1 - c0) < CH ? (t1 - c0) : CH);
        __syncthreads();  // previous chunk is done with LDS
        // ---- commit the prefetched chunk to LDS, then start fetching the next one
        pk.commit(sK, SK, KPL, nullptr, 0, 0, tid);
        if (with_out) pq.commit(sQ, SK, KPL, nullptr, 0, 0, tid);
        if (load_v) pv.commit(sV, SV, VPL, nullptr, 0, 0, tid);
        if (tid < CH) {
            sGr[tid] = pg;
            sBe[tid] = pb;
        }
        if (c0 + CH < t1) prefetch(c0 + CH);
        __syncthreads();

        // ---- in-chunk cumulative log-gate (every wave keeps its own copy)
        const float gc_l = wave_incl_scan(lane < CH ? sGr[lane] : 0.f, lane);
        sGc[lane] = gc_l;
        const float gtot = __shfl(gc_l, CH - 1, 64);
        lam_sum += gtot;
        wave_lds_sync();

        // ---- token x token products (shared by the workgroup)
        if (FAM == FAM_GDN || with_out) {
            constexpr int NPAIR = NTC * (NTC + 1) / 2;
            const int nprod = (FAM == FAM_GDN) ? (with_out ? 2 : 1) : 1;
            for (int item = w; item < nprod * NPAIR; item += NW) {
                const int which = item / NPAIR;  // GDN: 0 = K K^T, 1 = Q K^T; SSD: 0 = C B^T
                int pi = item % NPAIR, mt = 0;
                while (pi > mt) { pi -= mt + 1; ++mt; }
                const int nt = pi;
                const bool is_kk = (FAM == FAM_GDN) && which == 0;
                const bf16* A = is_kk ? sK : sQ;
                f32x4 acc = gemm_lds_lds<DK, F32IO>(A + (16 * mt + c16) * SK, A + KPL + (16 * mt + c16) * SK,
                                                    sK + (16 * nt + c16) * SK,
                                                    sK + KPL + (16 * nt + c16) * SK, g, zero4());
                const int i = 16 * nt + c16;
                const float gci = sGc[i];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = 16 * mt + 4 * g + r;
                    const float dec = __expf(sGc[t] - gci);
                    if (is_kk) {
                        sL[t * SCF + i] = (i < t) ? sBe[t] * dec * acc[r] : 0.f;
                    } else {
                        float v;
                        if (FAM == FAM_GDN) v = (i <= t) ? p.scale * dec * acc[r] : 0.f;
                        else v = (i <= t) ? dec * sBe[i] * acc[r] : 0.f;
                        const bf16 hi = (bf16)v;
                        sP[t * SC + i] = hi;
                        if (F32IO) sP[PPL + t * SC + i] = (bf16)(v - (float)hi);
                    }
                }
            }
            if (FAM == FAM_GDN) {
                __syncthreads();
                // inverse of each 16x16 diagonal block of (I + L): wave w, lane group
                // g handles block w + NW*g, lane c16 computes column c16
                const int b = w + NW * g;
                if (b < NTC) {
                    float x[16];
                    const float* Lb = sL + (16 * b) * SCF + 16 * b;
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        float acc = 0.f;
#pragma unroll
                        for (int m = 0; m < i; ++m) acc += Lb[i * SCF + m] * x[m];
                        x[i] = (i == c16) ? 1.f : (i < c16 ? 0.f : -acc);
                    }
#pragma unroll
                    for (int i = 0; i < 16; ++i) sN[b * 16 * SN + i * SN + c16] = x[i];
                }
            }
            __syncthreads();
        }

        // ---- per-wave state-row work (this lane's column = state row my_row)
        bf16x4 Sh[NTK], Sl[NTK];
#pragma unroll
        for (int nt = 0; nt < NTK; ++nt) {
            const Split4 sp = split4(S[nt]);
            Sh[nt] = sp.hi;
            Sl[nt] = sp.lo;
        }
        f32x4 U[NTC];
        bf16x4 Uh[NTC], Ul[NTC];
        if (FAM == FAM_GDN) {
            // X = V - diag(b) K S^T, then U = (I+L)^{-1} diag(beta) X by block substitution
#pragma unroll
            for (int mt = 0; mt < NTC; ++mt) {
                const bf16* kr = sK + (16 * mt + c16) * SK;
                f32x4 ks = gemm_lds_reg<F32IO, true>(kr, kr + KPL, Sh, Sl, 0, NTK, g, zero4());
                const f32x4 gct = lds4f(sGc + 16 * mt + 4 * g);
                const f32x4 bet = lds4f(sBe + 16 * mt + 4 * g);
                f32x4 vv = zero4();
                if (load_v) {
                    vv = to_f32(lds4_tr(sV, SV, 16 * mt, 16 * w, g, c16));
                    if (F32IO) vv += to_f32(lds4_tr(sV + VPL, SV, 16 * mt, 16 * w, g, c16));
                }
                f32x4 acc;
#pragma unroll
                for (int r = 0; r < 4; ++r) acc[r] = bet[r] * (vv[r] - __expf(gct[r]) * ks[r]);
                // subtract the coupling to earlier 16-token blocks: acc -= L[mt, <mt] U[<mt]
                acc = gemm_ldsf_reg<true>(sL + (16 * mt + c16) * SCF, Uh, Ul, 0, mt, g, acc);
                const Split4 rs = split4(acc);
                const float* nrow = sN + mt * 16 * SN + c16 * SN;
                U[mt] = gemm_ldsf_reg<false>(nrow, &rs.hi, &rs.lo, 0, 1, g, zero4());
                const Split4 us = split4(U[mt]);
                Uh[mt] = us.hi;
                Ul[mt] = us.lo;
            }
        } else {
#pragma unroll
            for (int mt = 0; mt < NTC; ++mt) {
                const bf16x4 xh = lds4_tr(sV, SV, 16 * mt, 16 * w, g, c16);
                U[mt] = to_f32(xh);
                Uh[mt] = xh;
                if (F32IO) {
                    const bf16x4 xl = lds4_tr(sV + VPL, SV, 16 * mt, 16 * w, g, c16);
                    U[mt] += to_f32(xl);
                    Ul[mt] = xl;
                } else {
                    Ul[mt] = bf16x4{(bf16)0.f, (bf16)0.f, (bf16)0.f, (bf16)0.f};
                }
            }
        }

        // ---- outputs
        if (with_out) {
#pragma unroll
            for (int mt = 0; mt < NTC; ++mt) {
                const bf16* qr = sQ + (16 * mt + c16) * SK;
                f32x4 qs = F32IO ? gemm_lds_reg<true, true>(qr, qr + KPL, Sh, Sl, 0, NTK, g, zero4())
                                 : gemm_lds_reg<false, false>(qr, qr, Sh, Sl, 0, NTK, g, zero4());
                const f32x4 gct = lds4f(sGc + 16 * mt + 4 * g);
                const float coef = (FAM == FAM_GDN) ? p.scale : 1.f;
                f32x4 o;
#pragma unroll
                for (int r = 0; r < 4; ++r) o[r] = coef * __expf(gct[r]) * qs[r];
                const bf16* pr = sP + (16 * mt + c16) * SC;
                o = F32IO ? gemm_lds_reg<true, true>(pr, pr + PPL, Uh, Ul, 0, mt + 1, g, o)
                          : gemm_lds_reg<false, false>(pr, pr, Uh, Ul, 0, mt + 1, g, o);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = 16 * mt + 4 * g + r;
                    if (t < n) {
                        const int64_t oi = ((c0 + t) * p.h_v + h) * (int64_t)p.dv + my_row;
                        if (F32IO) reinterpret_cast<float*>(p.out)[oi] = o[r];
                        else reinterpret_cast<bf16*>(p.out)[oi] = (bf16)o[r];
                    }
                }
            }
        }

        // ---- state update: S <- exp(gtot) S + K^T diag(w) U
        bf16x4 Wh[NTC], Wl[NTC];
#pragma unroll
        for (int mt = 0; mt < NTC; ++mt) {
            const f32x4 gct = lds4f(sGc + 16 * mt + 4 * g);
            f32x4 wu;
            if (FAM == FAM_GDN) {
#pragma unroll
                for (int r = 0; r < 4; ++r) wu[r] = __expf(gtot - gct[r]) * U[mt][r];
            } else {
                const f32x4 dt = lds4f(sBe + 16 * mt + 4 * g);
#pragma unroll
                for (int r = 0; r < 4; ++r) wu[r] = dt[r] * __expf(gtot - gct[r]) * U[mt][r];
            }
            const Split4 sp = split4(wu);
            Wh[mt] = sp.hi;
            Wl[mt] = sp.lo;
        }
        const float bC = __expf(gtot);
#pragma unroll
        for (int nt = 0; nt < NTK; ++nt) {
            S[nt] = gemm_ldstr_reg<F32IO, true>(sK, sK + KPL, SK, 16 * nt, Wh, Wl, 0, NTC, g, c16, bC * S[nt]);
        }
    }

    // ---- results
    float* dst = mtile ? p.M_out : p.S_final;
    if (dst) {
        const int rows = mtile ? DK : p.dv;
#pragma unroll
        for (int nt = 0; nt < NTK; ++nt)
            *reinterpret_cast<f32x4*>(dst + ((int64_t(s) * p.h_v + h) * rows + my_row) * DK + 16 * nt + 4 * g) =
                S[nt];
    }
    if (FAM == FAM_SSD && SUMMARY && p.M_out && tile == 0 && tid == 0)
        p.M_out[int64_t(s) * p.h_v + h] = lam_sum;
}

hipError_t launch_scan_gdn(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st);
hipError_t launch_scan_ssd(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st);
size_t scan_lds_bytes(int fam, int dk, int chunk, bool f32io, int nw, bool summary);

template <int FAM, int DK, int CH, bool F32IO, int NW, bool SUMMARY>
hipError_t launch_scan_nw(const ScanArgs& a, hipStream_t st) {
    const size_t lds = ScanLds<FAM, DK, CH, F32IO, NW>::bytes(SUMMARY);
    auto kern = scan_kernel<FAM, DK, CH, F32IO, NW, SUMMARY>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3(a.n_units), dim3(64 * NW), lds, st, a);
    return hipGetLastError();
}

template <int FAM, int DK, int CH, bool F32IO, bool SUMMARY>
hipError_t launch_scan_s(const ScanArgs& a, hipStream_t st) {
    switch (a.nw) {
        case 1: return launch_scan_nw<FAM, DK, CH, F32IO, 1, SUMMARY>(a, st);
        case 2: return launch_scan_nw<FAM, DK, CH, F32IO, 2, SUMMARY>(a, st);
        case 4: return launch_scan_nw<FAM, DK, CH, F32IO, 4, SUMMARY>(a, st);
    }
    return hipErrorInvalidValue;
}

// The block summary is its own instantiation (no output path, less LDS) and
// shows up under its own kernel name in traces.
template <int FAM, int DK, int CH, bool F32IO>
hipError_t launch_scan_t(const ScanArgs& a, hipStream_t st) {
    return a.summary ? launch_scan_s<FAM, DK, CH, F32IO, true>(a, st)
                     : launch_scan_s<FAM, DK, CH, F32IO, false>(a, st);
}

template <int FAM, int DK, int CH, bool F32IO>
size_t scan_lds_t(int nw, bool summary) {
    switch (nw) {
        case 1: return ScanLds<FAM, DK, CH, F32IO, 1>::bytes(summary);
        case 2: return ScanLds<FAM, DK, CH, F32IO, 2>::bytes(summary);
        case 4: return ScanLds<FAM, DK, CH, F32IO, 4>::bytes(summary);
    }
    return 0;
}

}  // namespace lkv
