// Chunkwise scan kernel for one recurrent layer (Gated DeltaNet or Mamba-2).
// Used by lkv_gdn_chunk_scan / lkv_ssd_chunk_scan (online prefill, outputs) and
// by lkv_block_summary (per-block state from zero, per-block transition).
//
// Work unit = (segment s, value head h, row tile of 16*NB state rows).  Rows of
// a dv x dk state evolve independently (the transition acts on the dk side),
// so splitting rows across workgroups is exact.
//
// Per chunk of CH tokens, with token rows Q, K (CH x dk), V (CH x dv),
// in-chunk cumulative log-gates gc_t (alpha_t = exp(g_t), Sec. 2), b_t =
// exp(gc_t) and w_t = exp(gc_C - gc_t), the block map of Eq. 5 applied to the
// chunk gives, for Gated DeltaNet (Eq. 3):
//   L = diag(beta) * strictly-lower(exp(gc_t - gc_i) * K K^T)
//   U = (I + L)^{-1} diag(beta) (V - diag(b) K S^T)              (delta-rule write)
//   O = scale (diag(b) Q S^T + lower(exp(gc_t - gc_i) * Q K^T) U)
//   S <- b_C S + U^T diag(w) K
// and for Mamba-2 (Eq. 2; q = C, k = B, v = x, gc = A_h * cumsum(dt)):
//   O = diag(b) C S^T + lower(exp(gc_t - gc_i) * C B^T) diag(dt) X
//   S <- b_C S + X^T diag(dt * w) B
//
// The work of a chunk splits into a state-independent part (gate prefix, the
// token x token products and masks, inverses of the 16x16 diagonal blocks of
// I + L) and the state chain.  The workgroup runs them as a two-stage
// software pipeline over chunks:
//   * A-waves (NA = 4): stage chunk c+1 from registers into LDS and prefetch
//     chunk c+2 from HBM; then compute chunk c+1's state-independent blocks,
//     stored pre-split (bf16 hi/lo) and transposed for direct fragment reads;
//   * B-waves (NB, 16 state rows each): chunk c's state chain -- K S^T, the
//     block forward substitution for U, the outputs, the state update -- with
//     the fp32 state held in MFMA accumulator registers throughout.
// LDS holds two pipeline buffers; two workgroup barriers per chunk.
//
// Precision: bf16 inputs enter the matrix cores exactly.  fp32 operands of the
// products that feed the state are split into bf16 hi + lo parts and
// multiplied as hi*hi + hi*lo + lo*hi (~2^-16 relative); products that only
// feed the bf16 output use the hi part.  With fp32 inputs every operand is
// split.
#pragma once
#include "frag_gemm.h"

namespace lkv {

enum { FAM_GDN = 0, FAM_SSD = 1 };
constexpr int NA = 4;  // A-waves per workgroup

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
    int32_t gate_bf16;   // GDN gates stored as bf16
    float scale;
    const float* S_init;  // scan: [n_seq,h_v,dv,dk] or null
    void* out;            // scan: o / y [n_tok,h_v,dv] or null
    float* S_final;       // scan: final state; summary: B_out (may be null)
    float* M_out;         // summary: GDN M [n_seq,h_v,dk,dk] / SSD Lambda [n_seq,h_v], or null
    int32_t summary;      // 0: scan from S_init with outputs; 1: block summary
    int32_t tiles_b;      // row tiles over dv (state rows)
    int32_t tiles_m;      // row tiles over dk (transition rows), GDN summary only
    int32_t nb;           // B-waves per workgroup (16*nb rows per tile)
    int32_t n_units;
};

template <int FAM, int DK, int CH, bool F32IO, int NB, bool SUMMARY>
struct ChunkLds {
    static constexpr int NTC = CH / 16;
    static constexpr int NOFF = NTC * (NTC - 1) / 2;  // strictly-lower 16x16 blocks
    static constexpr int NPB = NTC * (NTC + 1) / 2;   // lower blocks incl. the diagonal
    static constexpr int SK = DK + 8;                 // bf16 stride of [tok][dk] rows
    static constexpr int SV = 16 * NB + 8;            // bf16 stride of [tok][rows] rows
    static constexpr int SB = 20;                     // bf16 stride of a 16x16 block
    static constexpr int BLK = 16 * SB;               // elements per block plane
    static constexpr int SLD = 20;                    // f32 stride of the inverse scratch
    static constexpr int PL = F32IO ? 2 : 1;
    static constexpr bool HAS_Q = !SUMMARY;
    static constexpr bool HAS_L = FAM == FAM_GDN;
    static __host__ __device__ constexpr size_t al(size_t x) { return (x + 15) & ~size_t(15); }
    static constexpr size_t K_SZ = al(size_t(PL) * CH * SK * 2);
    static constexpr size_t Q_SZ = HAS_Q ? al(size_t(PL) * CH * SK * 2) : 0;
    static constexpr size_t V_SZ = al(size_t(PL) * CH * SV * 2);
    static constexpr size_t G_SZ = al((4 * CH + 4) * 4);
    static constexpr size_t LT_SZ = HAS_L ? al(size_t(NOFF) * BLK * 2 * 2) : 0;
    static constexpr size_t NT_SZ = HAS_L ? al(size_t(NTC) * BLK * 2 * 2) : 0;
    static constexpr size_t PT_SZ = HAS_Q ? al(size_t(NPB) * BLK * PL * 2) : 0;
    static constexpr size_t K_OFF = 0;
    static constexpr size_t Q_OFF = K_OFF + K_SZ;
    static constexpr size_t V_OFF = Q_OFF + Q_SZ;
    static constexpr size_t G_OFF = V_OFF + V_SZ;
    static constexpr size_t LT_OFF = G_OFF + G_SZ;
    static constexpr size_t NT_OFF = LT_OFF + LT_SZ;
    static constexpr size_t PT_OFF = NT_OFF + NT_SZ;
    static constexpr size_t BUF = PT_OFF + PT_SZ;  // one pipeline buffer
    static constexpr size_t GC_OFF = 2 * BUF;      // per A-wave gate prefix
    static constexpr size_t INV_OFF = GC_OFF + al(NA * 64 * 4);
    static constexpr size_t BYTES = INV_OFF + (HAS_L ? al(size_t(NA) * 16 * SLD * 4) : 0);
};

// index of block (mt, nt) among the strictly-lower blocks (nt < mt) / lower blocks (nt <= mt)
__device__ __forceinline__ constexpr int off_index(int mt, int nt) { return mt * (mt - 1) / 2 + nt; }
__device__ __forceinline__ constexpr int low_index(int mt, int nt) { return mt * (mt + 1) / 2 + nt; }

template <int FAM, int DK, int CH, bool F32IO, int NB, bool SUMMARY>
__global__ __launch_bounds__(64 * (NB + NA)) void chunk_kernel(ScanArgs p) {
    using Ly = ChunkLds<FAM, DK, CH, F32IO, NB, SUMMARY>;
    constexpr int NTC = CH / 16, NTK = DK / 16, NTHA = 64 * NA;
    constexpr int SK = Ly::SK, SV = Ly::SV, SB = Ly::SB, BLK = Ly::BLK, SLD = Ly::SLD;
    constexpr int NOFF = Ly::NOFF, NPB = Ly::NPB;
    constexpr int KPL = CH * SK, VPL = CH * SV;  // lo-plane offsets (fp32 io)
    extern __shared__ __align__(16) char smem[];

    const int tid = threadIdx.x;
    const int w = tid >> 6, lane = tid & 63, g = lane >> 4, c16 = lane & 15;
    const bool is_b = w < NB;
    const int wa = w - NB;            // A-wave index
    const int tid_a = tid - 64 * NB;  // thread index among the A-waves

    // ---- work unit
    const int tiles = p.tiles_b + p.tiles_m;
    const int u = xcd_unit(blockIdx.x, p.n_units);
    const int tile = u % tiles;
    const int h = (u / tiles) % p.h_v;
    const int s = u / (tiles * p.h_v);
    const bool mtile = tile >= p.tiles_b;
    const int row0 = (mtile ? tile - p.tiles_b : tile) * 16 * NB;
    const int my_row = row0 + 16 * w + c16;  // B-waves: this lane's state row
    const int hq = h / (p.h_v / p.h_qk);
    int64_t t0 = p.cu[s], t1 = p.cu[s + 1];
    t0 = t0 < 0 ? 0 : (t0 > p.n_tok ? p.n_tok : t0);
    t1 = t1 < t0 ? t0 : (t1 > p.n_tok ? p.n_tok : t1);
    const int nch = (int)((t1 - t0 + CH - 1) / CH);
    const bool with_out = !SUMMARY && p.out != nullptr;
    const bool load_v = !mtile;
    const float Ah = (FAM == FAM_SSD) ? p.A[h] : 0.f;

    auto sK = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::K_OFF); };
    auto sQ = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::Q_OFF); };
    auto sV = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::V_OFF); };
    auto sG = [&](int b) { return reinterpret_cast<float*>(smem + b * Ly::BUF + Ly::G_OFF); };
    auto sLT = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::LT_OFF); };
    auto sNT = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::NT_OFF); };
    auto sPT = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::PT_OFF); };

    // The two roles run separate loops with the same sequence of workgroup
    // barriers (s_barrier counts arriving waves, whatever the code location), so
    // each role's registers are allocated on its own: the B-waves' state and the
    // A-waves' prefetch registers never have to be live at the same time.
    if (is_b) {
        // ---- the state (acc layout: tile nt holds S[my_row][16nt + 4g + r])
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
        __syncthreads();  // prologue: chunk 0 staged by the A-waves
        for (int ci = 0; ci < nch; ++ci) {
            const int b = ci & 1;
            const int64_t c0 = t0 + (int64_t)ci * CH;
            const int n = (int)((t1 - c0) < CH ? (t1 - c0) : CH);
            __syncthreads();
            // ================= phase I: K S^T and the delta-rule right-hand side
            f32x4 X[NTC];
            bf16x4 Sh[NTK];
            {
                const bf16* Kb = sK(b);
                const float* G = sG(b);
                bf16x4 Sl[NTK];
#pragma unroll
                for (int nt = 0; nt < NTK; ++nt) {
                    const Split4 sp = split4(S[nt]);
                    Sh[nt] = sp.hi;
                    Sl[nt] = sp.lo;
                }
#pragma unroll
                for (int mt = 0; mt < NTC; ++mt) {
                    X[mt] = zero4();
                    if (load_v) {
                        X[mt] = to_f32(lds4_tr(sV(b), SV, 16 * mt, 16 * w, g, c16));
                        if (F32IO) X[mt] += to_f32(lds4_tr(sV(b) + VPL, SV, 16 * mt, 16 * w, g, c16));
                    }
                }
                if (FAM == FAM_GDN) {
                    // K S^T for all token tiles at once (interleaved chains, hi and lo passes apart)
                    f32x4 kh[NTC], kl[NTC];
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) kh[mt] = kl[mt] = zero4();
                    mgemm_rows<NTC, F32IO, true>(Kb + c16 * SK, 16 * SK, KPL, Sh, Sl, NTK, g, kh, kl);
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) {
                        const f32x4 bt = lds4f(G + 2 * CH + 16 * mt + 4 * g);
                        const f32x4 be = lds4f(G + CH + 16 * mt + 4 * g);
                        const f32x4 ks = kh[mt] + kl[mt];
#pragma unroll
                        for (int r = 0; r < 4; ++r) X[mt][r] = be[r] * (X[mt][r] - bt[r] * ks[r]);
                    }
                }
            }
            __syncthreads();
            // ================= phase II: substitution, outputs, state update
            {
                const bf16* Kb = sK(b);
                const float* G = sG(b);
                f32x4 U[NTC];
                bf16x4 Uh[NTC], Ul[NTC];
                if (FAM == FAM_GDN) {
                    // U_mt = N_mt (beta X_mt - sum_{m<mt} L_{mt,m} U_m)   (blocks of 16 tokens);
                    // the hi*hi and the correction passes accumulate apart
                    const bf16* LT = sLT(b);
                    const bf16* NT = sNT(b);
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) {
                        auto lhi = [&](int kg) { return LT + off_index(mt, kg) * BLK; };
                        auto llo = [&](int kg) { return LT + NOFF * BLK + off_index(mt, kg) * BLK; };
                        // hi*hi onto X; hi*lo and lo*hi in a second accumulator
                        const f32x4 a0 = gemm_blk_reg<SB, false, false>(lhi, 0, Uh, Uh, 0, mt, g, c16, X[mt]);
                        f32x4 a1 = gemm_blk_reg<SB, false, false>(lhi, 0, Ul, Ul, 0, mt, g, c16, zero4());
                        a1 = gemm_blk_reg<SB, false, false>(llo, 0, Uh, Uh, 0, mt, g, c16, a1);
                        const Split4 rs = split4(a0 + a1);
                        const bf16* nb = NT + mt * BLK;
                        const bf16x4 nh = lds4_tr(nb, SB, 0, 0, g, c16), nl = lds4_tr(nb + NTC * BLK, SB, 0, 0, g, c16);
                        f32x4 u0 = mma16(nh, rs.hi, zero4());
                        f32x4 u1 = mma16(nh, rs.lo, zero4());
                        u1 = mma16(nl, rs.hi, u1);
                        U[mt] = u0 + u1;
                        const Split4 us = split4(U[mt]);
                        Uh[mt] = us.hi;
                        Ul[mt] = us.lo;
                    }
                } else {
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) {
                        U[mt] = X[mt];
                        Uh[mt] = lds4_tr(sV(b), SV, 16 * mt, 16 * w, g, c16);
                        Ul[mt] = F32IO ? lds4_tr(sV(b) + VPL, SV, 16 * mt, 16 * w, g, c16) : zero_bf16x4();
                    }
                }
                if (with_out) {
                    const bf16* PT = sPT(b);
                    bf16x4 Sl[NTK];
                    if (F32IO) {
#pragma unroll
                        for (int nt = 0; nt < NTK; ++nt) Sl[nt] = to_bf16(S[nt] - to_f32(Sh[nt]));
                    }
                    const float coef = (FAM == FAM_GDN) ? p.scale : 1.f;
                    // Q S^T for all token tiles (interleaved), then the masked P U term
                    f32x4 qh[NTC], ql[NTC];
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) qh[mt] = ql[mt] = zero4();
                    mgemm_rows<NTC, F32IO, F32IO>(sQ(b) + c16 * SK, 16 * SK, KPL, Sh, Sl, NTK, g, qh, ql);
                    f32x4 O[NTC];
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) {
                        const f32x4 bt = lds4f(G + 2 * CH + 16 * mt + 4 * g);
                        const f32x4 qs = F32IO ? qh[mt] + ql[mt] : qh[mt];
#pragma unroll
                        for (int r = 0; r < 4; ++r) O[mt][r] = coef * bt[r] * qs[r];
                    }
                    // P U: tile mt contracts over token blocks 0..mt; pair index outer, tiles inner
                    if (NTC == 1) {
                        const bf16x4 x = lds4_tr(PT, SB, 0, 0, g, c16);
                        O[0] = mma16(x, Uh[0], O[0]);
                        if (F32IO) {
                            O[0] = mma16(x, Ul[0], O[0]);
                            O[0] = mma16(lds4_tr(PT + NPB * BLK, SB, 0, 0, g, c16), Uh[0], O[0]);
                        }
                    } else {
#pragma unroll
                        for (int kp = 0; kp < NTC; kp += 2) {
#pragma unroll
                            for (int mt = 0; mt < NTC; ++mt) {
                                if (mt < kp) continue;
                                const bool two = mt >= kp + 1;
                                const bf16* x0p = PT + low_index(mt, kp) * BLK;
                                const bf16x4 x0 = lds4_tr(x0p, SB, 0, 0, g, c16);
                                const bf16x4 x1 = two ? lds4_tr(x0p + BLK, SB, 0, 0, g, c16) : zero_bf16x4();
                                const bf16x4 u1h = two ? Uh[kp + 1] : zero_bf16x4();
                                O[mt] = mma32(x0, x1, Uh[kp], u1h, O[mt]);
                                if (F32IO) {
                                    const bf16x4 u1l = two ? Ul[kp + 1] : zero_bf16x4();
                                    O[mt] = mma32(x0, x1, Ul[kp], u1l, O[mt]);
                                    const bf16x4 y0 = lds4_tr(x0p + NPB * BLK, SB, 0, 0, g, c16);
                                    const bf16x4 y1 = two ? lds4_tr(x0p + NPB * BLK + BLK, SB, 0, 0, g, c16)
                                                          : zero_bf16x4();
                                    O[mt] = mma32(y0, y1, Uh[kp], u1h, O[mt]);
                                }
                            }
                        }
                    }
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) {
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const int t = 16 * mt + 4 * g + r;
                            if (t < n) {
                                const int64_t oi = ((c0 + t) * p.h_v + h) * (int64_t)p.dv + my_row;
                                if (F32IO) reinterpret_cast<float*>(p.out)[oi] = O[mt][r];
                                else reinterpret_cast<bf16*>(p.out)[oi] = (bf16)O[mt][r];
                            }
                        }
                    }
                }
                // S <- b_C S + K^T diag(w) U   (all dk tiles interleaved)
                bf16x4 Wh[NTC], Wl[NTC];
#pragma unroll
                for (int mt = 0; mt < NTC; ++mt) {
                    const f32x4 wt = lds4f(G + 3 * CH + 16 * mt + 4 * g);
                    const Split4 sp = split4(wt * U[mt]);
                    Wh[mt] = sp.hi;
                    Wl[mt] = sp.lo;
                }
                const float bC = G[4 * CH];
#pragma unroll
                for (int nt = 0; nt < NTK; ++nt) S[nt] = bC * S[nt];
                mgemm_tr<NTK, F32IO, true>(Kb, KPL, SK, Wh, Wl, NTC, g, c16, S);
            }
        }
        float* dst = mtile ? p.M_out : p.S_final;
        if (dst) {
            const int rows = mtile ? DK : p.dv;
#pragma unroll
            for (int nt = 0; nt < NTK; ++nt)
                *reinterpret_cast<f32x4*>(dst + ((int64_t(s) * p.h_v + h) * rows + my_row) * DK + 16 * nt + 4 * g) =
                    S[nt];
        }
    } else {
        // ---- A-waves: HBM -> register prefetch and register -> LDS commit of a chunk
        TileRegs<CH, DK, F32IO, NTHA> pk, pq;
        TileRegs<CH, 16 * NB, F32IO, NTHA> pv;
        uint32_t pg = 0u, pb = 0u;  // gates stay raw bits until commit (no early wait on the loads)
        float lam_sum = 0.f;
        constexpr int ES = F32IO ? 4 : 2;
        const uint32_t qk_rb = (uint32_t)(p.h_qk * DK * ES), v_rb = (uint32_t)(p.h_v * p.dv * ES);
        auto prefetch = [&](int ci) {
            const int64_t c0 = t0 + (int64_t)ci * CH;
            const int n = (int)((t1 - c0) < CH ? (t1 - c0) : CH);
            const int64_t qk_off = (c0 * p.h_qk + hq) * (int64_t)DK * ES;
            pk.load(reinterpret_cast<const char*>(p.k) + qk_off, qk_rb, n, tid_a);
            if (with_out) pq.load(reinterpret_cast<const char*>(p.q) + qk_off, qk_rb, n, tid_a);
            if (load_v)
                pv.load(reinterpret_cast<const char*>(p.v) + ((c0 * p.h_v + h) * (int64_t)p.dv + row0) * ES, v_rb, n,
                        tid_a);
            if (tid_a < CH) {
                const int64_t gi = (c0 + tid_a) * p.h_v + h;
                pg = pb = 0u;
                if (tid_a < n) {
                    if (FAM == FAM_GDN && p.gate_bf16) {
                        pg = reinterpret_cast<const uint16_t*>(p.g)[gi];
                        pb = reinterpret_cast<const uint16_t*>(p.beta)[gi];
                    } else if (FAM == FAM_GDN) {
                        pg = reinterpret_cast<const uint32_t*>(p.g)[gi];
                        pb = reinterpret_cast<const uint32_t*>(p.beta)[gi];
                    } else {
                        pg = reinterpret_cast<const uint32_t*>(p.g)[gi];  // dt
                    }
                }
            }
        };
        auto commit = [&](int ci) {
            const int b = ci & 1;
            pk.commit(sK(b), SK, KPL, tid_a);
            if (with_out) pq.commit(sQ(b), SK, KPL, tid_a);
            if (load_v) pv.commit(sV(b), SV, VPL, tid_a);
            if (tid_a < CH) {
                float* G = sG(b);
                const bool b16 = FAM == FAM_GDN && p.gate_bf16;
                G[tid_a] = __builtin_bit_cast(float, b16 ? pg << 16 : pg);
                G[CH + tid_a] = __builtin_bit_cast(float, b16 ? pb << 16 : pb);
            }
        };

        // A-waves: state-independent blocks of chunk ci into buffer ci & 1
        auto a_work = [&](int ci) {
            const int b = ci & 1;
            float* G = sG(b);
            const bf16* Kb = sK(b);
            const bf16* Qb = sQ(b);
            float* gcw = reinterpret_cast<float*>(smem + Ly::GC_OFF) + 64 * wa;
            // in-chunk cumulative log-gate, lane = token
            const float gate = lane < CH ? (FAM == FAM_GDN ? G[lane] : Ah * G[lane]) : 0.f;
            const float gc = wave_incl_scan(gate, lane);
            const float gtot = __shfl(gc, CH - 1, 64);
            gcw[lane] = gc;
            if (wa == 0) {
                if (lane < CH) {
                    G[2 * CH + lane] = __expf(gc);
                    const float wt = __expf(gtot - gc);
                    G[3 * CH + lane] = (FAM == FAM_GDN) ? wt : G[lane] * wt;
                }
                if (lane == 0) {
                    G[4 * CH] = __expf(gtot);
                    G[4 * CH + 1] = gtot;
                }
                lam_sum += gtot;
            }
            wave_lds_sync();
            // Gated DeltaNet: inverse of diagonal block wa of (I + L)
            if (FAM == FAM_GDN && wa < NTC) {
                const int mt = wa;
                const bf16* kr = Kb + (16 * mt + c16) * SK;
                const f32x4 acc = gemm_lds_lds<DK, F32IO>(kr, kr + KPL, kr, kr + KPL, g, zero4());
                float* LTd = reinterpret_cast<float*>(smem + Ly::INV_OFF) + wa * 16 * SLD;
                const float gci = gcw[16 * mt + c16];
                f32x4 l;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = 4 * g + r;  // local row; column c16
                    l[r] = (c16 < t) ? G[CH + 16 * mt + t] * __expf(gcw[16 * mt + t] - gci) * acc[r] : 0.f;
                }
                *reinterpret_cast<f32x4*>(LTd + c16 * SLD + 4 * g) = l;  // LTd[i][t] = L[t][i]
                wave_lds_sync();
                // column c16 of (I + L_mm)^{-1}, right-looking forward substitution; each
                // finished entry goes straight to NT[c16][m] = N[m][c16] (bf16 hi / lo)
                bf16* nt_hi = sNT(b) + mt * BLK + c16 * SB;
                bf16* nt_lo = nt_hi + NTC * BLK;
                // the whole block in registers first (columns of L are rows of LTd), so the
                // 16 dependent steps below wait on FMAs only, not on LDS
                f32x4 Lc[15][4];
#pragma unroll
                for (int m = 0; m < 15; ++m)
#pragma unroll
                    for (int q4 = (m + 1) >> 2; q4 < 4; ++q4) Lc[m][q4] = lds4f(LTd + m * SLD + 4 * q4);
                float a[16];
#pragma unroll
                for (int i = 0; i < 16; ++i) a[i] = 0.f;
#pragma unroll
                for (int m = 0; m < 16; ++m) {
                    const float xm = (m == c16) ? 1.f : (m < c16 ? 0.f : -a[m]);
                    if (g == 0) {
                        const bf16 hi = (bf16)xm;
                        nt_hi[m] = hi;
                        nt_lo[m] = (bf16)(xm - (float)hi);
                    }
                    if (m < 15) {
#pragma unroll
                        for (int i = m + 1; i < 16; ++i) a[i] += Lc[m][i >> 2][i & 3] * xm;
                    }
                }
            }
            // token x token blocks: GDN strictly-lower K K^T blocks (negated L), then the
            // output blocks Q K^T (GDN) / C B^T (SSD)
            constexpr int N_OFFI = (FAM == FAM_GDN) ? NOFF : 0;
            const int n_items = N_OFFI + (with_out ? NPB : 0);
            for (int j = wa; j < n_items; j += NA) {
                const bool is_l = j < N_OFFI;
                int mt, nt;
                if (is_l) {
                    mt = 1;
                    while (off_index(mt + 1, 0) <= j) ++mt;
                    nt = j - off_index(mt, 0);
                } else {
                    const int jj = j - N_OFFI;
                    mt = 0;
                    while (low_index(mt + 1, 0) <= jj) ++mt;
                    nt = jj - low_index(mt, 0);
                }
                const bf16* A = is_l ? Kb : Qb;
                const bf16* ar = A + (16 * mt + c16) * SK;
                const bf16* br = Kb + (16 * nt + c16) * SK;
                const f32x4 acc = gemm_lds_lds<DK, F32IO>(ar, ar + KPL, br, br + KPL, g, zero4());
                const int i = 16 * nt + c16;
                const float gci = gcw[i];
                f32x4 v;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = 16 * mt + 4 * g + r;
                    const float dec = __expf(gcw[t] - gci);
                    if (is_l) v[r] = -G[CH + t] * dec * acc[r];  // nt < mt: every entry is below the diagonal
                    else if (FAM == FAM_GDN) v[r] = (i <= t) ? p.scale * dec * acc[r] : 0.f;
                    else v[r] = (i <= t) ? G[i] * dec * acc[r] : 0.f;
                }
                if (is_l) {
                    store_tile_tr<SB, true>(sLT(b) + off_index(mt, nt) * BLK, NOFF * BLK, v, g, c16);
                } else {
                    store_tile_tr<SB, F32IO>(sPT(b) + low_index(mt, nt) * BLK, NPB * BLK, v, g, c16);
                }
            }
        };

        // prologue: chunk 0 staged and its blocks built; chunk 1 in flight.  Chunk
        // c+1's loads are issued at the END of phase II and committed at the start
        // of the next phase I, so they overlap the B-waves' remaining work.
        if (nch > 0) {
            prefetch(0);
            commit(0);
        }
        __syncthreads();
        if (nch > 0) {
            a_work(0);
            if (nch > 1) prefetch(1);
        }
        for (int ci = 0; ci < nch; ++ci) {
            __syncthreads();
            if (ci + 1 < nch) commit(ci + 1);
            __syncthreads();
            if (ci + 1 < nch) {
                a_work(ci + 1);
                if (ci + 2 < nch) prefetch(ci + 2);
            }
        }
        if (FAM == FAM_SSD && SUMMARY && p.M_out && tile == 0 && wa == 0 && lane == 0)
            p.M_out[int64_t(s) * p.h_v + h] = lam_sum;
    }
}

hipError_t launch_scan_gdn(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st);
hipError_t launch_scan_ssd(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st);
size_t scan_lds_bytes(int fam, int dk, int chunk, bool f32io, int nb, bool summary);

template <int FAM, int DK, int CH, bool F32IO, int NB, bool SUMMARY>
hipError_t launch_chunk_nb(const ScanArgs& a, hipStream_t st) {
    const size_t lds = ChunkLds<FAM, DK, CH, F32IO, NB, SUMMARY>::BYTES;
    auto kern = chunk_kernel<FAM, DK, CH, F32IO, NB, SUMMARY>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3(a.n_units), dim3(64 * (NB + NA)), lds, st, a);
    return hipGetLastError();
}

template <int FAM, int DK, int CH, bool F32IO, bool SUMMARY>
hipError_t launch_chunk_s(const ScanArgs& a, hipStream_t st) {
    switch (a.nb) {
        case 1: return launch_chunk_nb<FAM, DK, CH, F32IO, 1, SUMMARY>(a, st);
        case 2: return launch_chunk_nb<FAM, DK, CH, F32IO, 2, SUMMARY>(a, st);
        case 4: return launch_chunk_nb<FAM, DK, CH, F32IO, 4, SUMMARY>(a, st);
    }
    return hipErrorInvalidValue;
}

// The block summary is its own instantiation (no output path, less LDS) and
// shows up under its own kernel name in traces.
template <int FAM, int DK, int CH, bool F32IO>
hipError_t launch_chunk_t(const ScanArgs& a, hipStream_t st) {
    return a.summary ? launch_chunk_s<FAM, DK, CH, F32IO, true>(a, st)
                     : launch_chunk_s<FAM, DK, CH, F32IO, false>(a, st);
}

template <int FAM, int DK, int CH, bool F32IO>
size_t chunk_lds_t(int nb, bool summary) {
    switch (nb * 2 + (summary ? 1 : 0)) {
        case 2: return ChunkLds<FAM, DK, CH, F32IO, 1, false>::BYTES;
        case 3: return ChunkLds<FAM, DK, CH, F32IO, 1, true>::BYTES;
        case 4: return ChunkLds<FAM, DK, CH, F32IO, 2, false>::BYTES;
        case 5: return ChunkLds<FAM, DK, CH, F32IO, 2, true>::BYTES;
        case 8: return ChunkLds<FAM, DK, CH, F32IO, 4, false>::BYTES;
        case 9: return ChunkLds<FAM, DK, CH, F32IO, 4, true>::BYTES;
    }
    return 0;
}

}  // namespace lkv
