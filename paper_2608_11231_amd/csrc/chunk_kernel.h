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
#include <type_traits>

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
    // bf16 stride of [tok][dk] rows (kq_pos order): 16-byte aligned rows whose
    // fragment reads (16-byte row runs and transposed 8-byte reads) are free of
    // LDS bank conflicts
    static constexpr int SK = DK >= 32 ? DK + 16 : DK + 8;
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
    // gate rows: raw gate | beta | b | w | cumulative gate gc | b_C, gc_C
    static constexpr size_t G_SZ = al((5 * CH + 4) * 4);
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
    static constexpr int INV_BST = 16 * SLD + 4;      // f32 stride of inverse scratch blocks (bank shift)
    static constexpr size_t BYTES = INV_OFF + (HAS_L ? al(size_t(NTC) * INV_BST * 4) : 0);
};

// index of block (mt, nt) among the strictly-lower blocks (nt < mt) / lower blocks (nt <= mt)
__device__ __forceinline__ constexpr int off_index(int mt, int nt) { return mt * (mt - 1) / 2 + nt; }
__device__ __forceinline__ constexpr int low_index(int mt, int nt) { return mt * (mt + 1) / 2 + nt; }
// row block of the j-th strictly-lower / lower block in that order
__device__ __forceinline__ constexpr int off_mt(int j) {
    int mt = 1;
    while (off_index(mt + 1, 0) <= j) ++mt;
    return mt;
}
__device__ __forceinline__ constexpr int low_mt(int j) {
    int mt = 0;
    while (low_index(mt + 1, 0) <= j) ++mt;
    return mt;
}

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
    const bool load_v = SUMMARY ? !mtile : true;  // transition (M) tiles of a block summary skip V
    const float Ah = (FAM == FAM_SSD) ? p.A[h] : 0.f;

    auto sK = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::K_OFF); };
    auto sQ = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::Q_OFF); };
    auto sV = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::V_OFF); };
    auto sG = [&](int b) { return reinterpret_cast<float*>(smem + b * Ly::BUF + Ly::G_OFF); };
    auto sLT = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::LT_OFF); };
    auto sNT = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::NT_OFF); };
    auto sPT = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::PT_OFF); };

    // ---- state-independent token blocks of one chunk (buffer b).  Items are the
    // 16x16 blocks: the strictly-lower K K^T blocks of Gated DeltaNet (kind L,
    // stored negated as -L, hi / lo) and the lower Q K^T / C B^T output blocks
    // (kind P).  A wave takes items SLOT, SLOT + NSLOT, ... of one kind, fixed at
    // compile time, so all of its products run as independent accumulation
    // chains.  gcp: the chunk's cumulative log-gates.
    constexpr int NK = DK / 16;
    auto items = [&](auto slot_c, auto nslot_c, auto kind_l_c, int b, const float* gcp) {
        constexpr int SLOT = decltype(slot_c)::value;
        constexpr int NSLOT = decltype(nslot_c)::value;
        constexpr bool KL = decltype(kind_l_c)::value;
        constexpr int NIT = KL ? (FAM == FAM_GDN ? NOFF : 0) : (SUMMARY ? 0 : NPB);
        constexpr int NMY = NIT > SLOT ? (NIT - SLOT + NSLOT - 1) / NSLOT : 0;
        if constexpr (NMY > 0) {
            const bf16* Kb = sK(b);
            const bf16* Ab = KL ? sK(b) : sQ(b);
            const float* G = sG(b);
            auto item_mt = [](int i) { return KL ? off_mt(SLOT + i * NSLOT) : low_mt(SLOT + i * NSLOT); };
            auto item_nt = [](int i) {
                const int j = SLOT + i * NSLOT;
                return KL ? j - off_index(off_mt(j), 0) : j - low_index(low_mt(j), 0);
            };
            f32x4 acc[NMY];
#pragma unroll
            for (int i = 0; i < NMY; ++i) acc[i] = zero4();
            if constexpr (NK == 1) {
#pragma unroll
                for (int i = 0; i < NMY; ++i) {
                    const bf16* ar = Ab + (16 * item_mt(i) + c16) * SK + 4 * g;
                    const bf16* br = Kb + (16 * item_nt(i) + c16) * SK + 4 * g;
                    acc[i] = mma16(lds4(ar), lds4(br), acc[i]);
                    if (F32IO) {
                        acc[i] = mma16(lds4(ar), lds4(br + KPL), acc[i]);
                        acc[i] = mma16(lds4(ar + KPL), lds4(br), acc[i]);
                    }
                }
            } else {
                // fragments of slice kp+1 are requested before the products of slice kp
                constexpr int NKP = NK / 2, FPL = F32IO ? 2 : 1;
                bf16x8 fa[2][FPL][NMY], fb[2][FPL][NMY];
                auto fetch = [&](int kp, int buf) {
#pragma unroll
                    for (int i = 0; i < NMY; ++i) {
                        const bf16* ar = Ab + (16 * item_mt(i) + c16) * SK + 32 * kp + 8 * g;
                        const bf16* br = Kb + (16 * item_nt(i) + c16) * SK + 32 * kp + 8 * g;
#pragma unroll
                        for (int pl = 0; pl < FPL; ++pl) {
                            fa[buf][pl][i] = lds8(ar + pl * KPL);
                            fb[buf][pl][i] = lds8(br + pl * KPL);
                        }
                    }
                };
                fetch(0, 0);
#pragma unroll
                for (int kp = 0; kp < NKP; ++kp) {
                    const int cb = kp & 1;
                    if (kp + 1 < NKP) fetch(kp + 1, cb ^ 1);
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int i = 0; i < NMY; ++i) {
                        acc[i] = mma32(fa[cb][0][i], fb[cb][0][i], acc[i]);
                        if constexpr (F32IO) {
                            acc[i] = mma32(fa[cb][0][i], fb[cb][FPL - 1][i], acc[i]);
                            acc[i] = mma32(fa[cb][FPL - 1][i], fb[cb][0][i], acc[i]);
                        }
                    }
                }
            }
#pragma unroll
            for (int i = 0; i < NMY; ++i) {
                const int mt = item_mt(i), nt = item_nt(i);
                const int ic = 16 * nt + c16;
                const float gci = gcp[ic];
                const f32x4 gt = lds4f(gcp + 16 * mt + 4 * g);
                f32x4 v;
                if constexpr (KL) {
                    const f32x4 bt = lds4f(G + CH + 16 * mt + 4 * g);
#pragma unroll
                    for (int r = 0; r < 4; ++r) v[r] = -bt[r] * __expf(gt[r] - gci) * acc[i][r];
                    store_tile_tr<SB, true>(sLT(b) + off_index(mt, nt) * BLK, NOFF * BLK, v, g, c16);
                } else {
                    const float cf = (FAM == FAM_GDN) ? p.scale : G[ic];  // SSD: dt of column i
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float e = cf * __expf(gt[r] - gci) * acc[i][r];
                        v[r] = (mt > nt || c16 <= 4 * g + r) ? e : 0.f;
                    }
                    store_tile_tr<SB, F32IO>(sPT(b) + low_index(mt, nt) * BLK, NPB * BLK, v, g, c16);
                }
            }
        }
    };
    using std::integral_constant;
    using L_KIND = std::true_type;
    using P_KIND = std::false_type;

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
        // bf16 hi / lo parts of the state, refreshed after every state update
        bf16x4 Sh[NTK], Sl[NTK];
        auto split_state = [&]() {
#pragma unroll
            for (int nt = 0; nt < NTK; ++nt) {
                const Split4 sp = split4(S[nt]);
                Sh[nt] = sp.hi;
                Sl[nt] = sp.lo;
            }
        };
        split_state();
        __syncthreads();  // prologue: chunk 0 staged by the A-waves
        for (int ci = 0; ci < nch; ++ci) {
            const int b = ci & 1;
            const int64_t c0 = t0 + (int64_t)ci * CH;
            const int n = (int)((t1 - c0) < CH ? (t1 - c0) : CH);
            __syncthreads();
            // ================= phase I: K S^T and the delta-rule right-hand side
            f32x4 X[NTC];
            {
                const bf16* Kb = sK(b);
                const float* G = sG(b);
#pragma unroll
                for (int mt = 0; mt < NTC; ++mt) {
                    X[mt] = zero4();
                    if (load_v) {
                        X[mt] = to_f32(lds4_tr(sV(b), SV, 16 * mt, 16 * w, g, c16));
                        if (F32IO) X[mt] += to_f32(lds4_tr(sV(b) + VPL, SV, 16 * mt, 16 * w, g, c16));
                    }
                }
                if (with_out) {
                    // this chunk's output blocks P, shared by the B-waves (read after the barrier)
                    using NS = integral_constant<int, NB>;
                    const float* gcp = G + 4 * CH;
                    switch (w) {
                        case 0: items(integral_constant<int, 0>(), NS(), P_KIND(), b, gcp); break;
                        case 1: items(integral_constant<int, 1 % NB>(), NS(), P_KIND(), b, gcp); break;
                        case 2: items(integral_constant<int, 2 % NB>(), NS(), P_KIND(), b, gcp); break;
                        default: items(integral_constant<int, 3 % NB>(), NS(), P_KIND(), b, gcp); break;
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
                // Outputs are formed transposed, O^T = S Q^T + U^T P^T: tile mt holds
                // O[16mt + c16][this wave's rows 4g..4g+3], so each lane stores 4
                // consecutive state rows of one token.  S Q^T does not depend on U and
                // is issued first, alongside the substitution chain.
                f32x4 OT[NTC];
                if (with_out) {
                    const bf16* Qb = sQ(b);
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) OT[mt] = zero4();
                    if constexpr (NTK == 1) {
#pragma unroll
                        for (int mt = 0; mt < NTC; ++mt) {
                            const bf16* qr = Qb + (16 * mt + c16) * SK + 4 * g;
                            OT[mt] = mma16(Sh[0], lds4(qr), OT[mt]);
                            if (F32IO) {
                                OT[mt] = mma16(Sl[0], lds4(qr), OT[mt]);
                                OT[mt] = mma16(Sh[0], lds4(qr + KPL), OT[mt]);
                            }
                        }
                    } else {
                        constexpr int NKP = NTK / 2;
                        bf16x8 qh[NKP][NTC], ql[F32IO ? NKP : 1][NTC];
#pragma unroll
                        for (int kp = 0; kp < NKP; ++kp)
#pragma unroll
                            for (int mt = 0; mt < NTC; ++mt) {
                                const bf16* qr = Qb + (16 * mt + c16) * SK + 32 * kp + 8 * g;
                                qh[kp][mt] = lds8(qr);
                                if constexpr (F32IO) ql[kp][mt] = lds8(qr + KPL);
                            }
                        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                        for (int kp = 0; kp < NKP; ++kp)
#pragma unroll
                            for (int mt = 0; mt < NTC; ++mt) {
                                OT[mt] = mma32(Sh[2 * kp], Sh[2 * kp + 1], qh[kp][mt], OT[mt]);
                                if constexpr (F32IO) {
                                    OT[mt] = mma32(Sl[2 * kp], Sl[2 * kp + 1], qh[kp][mt], OT[mt]);
                                    OT[mt] = mma32(Sh[2 * kp], Sh[2 * kp + 1], ql[kp][mt], OT[mt]);
                                }
                            }
                    }
                }
                f32x4 U[NTC];
                bf16x4 Uh[NTC], Ul[NTC];
                // output blocks P (transposed fragments), independent of U: requested early
                constexpr int PPL = (!SUMMARY && F32IO) ? 2 : 1;
                bf16x4 Pf[PPL][SUMMARY ? 1 : NPB];
                if (with_out) {
#pragma unroll
                    for (int j = 0; j < NPB; ++j)
#pragma unroll
                        for (int pl = 0; pl < PPL; ++pl)
                            Pf[pl][j] = lds4_tr(sPT(b) + pl * NPB * BLK + j * BLK, SB, 0, 0, g, c16);
                }
                if (FAM == FAM_GDN) {
                    // U_mt = N_mt (beta X_mt - sum_{m<mt} L_{mt,m} U_m)   (blocks of 16 tokens);
                    // the hi*hi and the correction passes accumulate apart.  All L and N
                    // fragments are in registers before the dependent chain starts.
                    const bf16* LT = sLT(b);
                    const bf16* NT = sNT(b);
                    bf16x4 Lh[NOFF > 0 ? NOFF : 1], Ll[NOFF > 0 ? NOFF : 1], Nh[NTC], Nl[NTC];
#pragma unroll
                    for (int j = 0; j < NOFF; ++j) {
                        Lh[j] = lds4_tr(LT + j * BLK, SB, 0, 0, g, c16);
                        Ll[j] = lds4_tr(LT + (NOFF + j) * BLK, SB, 0, 0, g, c16);
                    }
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) {
                        Nh[mt] = lds4_tr(NT + mt * BLK, SB, 0, 0, g, c16);
                        Nl[mt] = lds4_tr(NT + (NTC + mt) * BLK, SB, 0, 0, g, c16);
                    }
                    // sum over token blocks kg < mt of A_{mt,kg} B_kg: pairs through the
                    // 32-wide MFMA, a lone block through the 16-wide one, an odd tail after
                    // pairs zero-padded (one shape per chain)
                    auto blk_sum = [&](const bf16x4* A, const bf16x4* B, int mt, f32x4 acc) {
                        int kg = 0;
#pragma unroll
                        for (; kg + 1 < mt; kg += 2)
                            acc = mma32(A[off_index(mt, kg)], A[off_index(mt, kg + 1)], B[kg], B[kg + 1], acc);
                        if (kg < mt) {
                            if (kg == 0) {
                                acc = mma16(A[off_index(mt, kg)], B[kg], acc);
                            } else {
                                const bf16x4 z = zero_bf16x4();
                                acc = mma32(A[off_index(mt, kg)], z, B[kg], z, acc);
                            }
                        }
                        return acc;
                    };
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) {
                        const f32x4 a0 = blk_sum(Lh, Uh, mt, X[mt]);
                        f32x4 a1 = blk_sum(Lh, Ul, mt, zero4());
                        a1 = blk_sum(Ll, Uh, mt, a1);
                        const Split4 rs = split4(a0 + a1);
                        const bf16x4 nh = Nh[mt], nl = Nl[mt];
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
                    const float coef = (FAM == FAM_GDN) ? p.scale : 1.f;
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) OT[mt] *= coef * G[2 * CH + 16 * mt + c16];
                    // + U^T P^T: tile mt contracts over token blocks 0..mt, pairs of blocks per MFMA
                    if constexpr (NTC == 1) {
                        const bf16x4 x = Pf[0][0];
                        OT[0] = mma16(Uh[0], x, OT[0]);
                        if (F32IO) {
                            OT[0] = mma16(Ul[0], x, OT[0]);
                            OT[0] = mma16(Uh[0], Pf[PPL - 1][0], OT[0]);
                        }
                    } else {
#pragma unroll
                        for (int kp = 0; kp < NTC; kp += 2) {
#pragma unroll
                            for (int mt = 0; mt < NTC; ++mt) {
                                if (mt < kp) continue;
                                const bool two = mt >= kp + 1;
                                const int j0 = low_index(mt, kp);
                                const bf16x4 x0 = Pf[0][j0];
                                const bf16x4 x1 = two ? Pf[0][j0 + 1] : zero_bf16x4();
                                const bf16x4 u1h = two ? Uh[kp + 1] : zero_bf16x4();
                                OT[mt] = mma32(Uh[kp], u1h, x0, x1, OT[mt]);
                                if (F32IO) {
                                    const bf16x4 u1l = two ? Ul[kp + 1] : zero_bf16x4();
                                    OT[mt] = mma32(Ul[kp], u1l, x0, x1, OT[mt]);
                                    const bf16x4 y0 = Pf[PPL - 1][j0];
                                    const bf16x4 y1 = two ? Pf[PPL - 1][j0 + 1] : zero_bf16x4();
                                    OT[mt] = mma32(Uh[kp], u1h, y0, y1, OT[mt]);
                                }
                            }
                        }
                    }
                    // one 8-byte (bf16) / 16-byte (fp32) store per lane and token tile
                    const int64_t rowcol = (int64_t)h * p.dv + row0 + 16 * w + 4 * g;
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) {
                        const int t = 16 * mt + c16;
                        if (t < n) {
                            const int64_t oi = (c0 + t) * p.h_v * (int64_t)p.dv + rowcol;
                            if (F32IO) *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(p.out) + oi) = OT[mt];
                            else *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(p.out) + oi) = to_bf16(OT[mt]);
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
                const float bC = G[5 * CH];
#pragma unroll
                for (int nt = 0; nt < NTK; ++nt) S[nt] = bC * S[nt];
                mgemm_tr<DK, NTK, F32IO, true>(Kb, KPL, SK, Wh, Wl, NTC, g, c16, S);
                split_state();  // for the next chunk, ahead of its barrier
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
        KQTile<CH, DK, F32IO, NTHA> pk, pq;
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

        // Gated DeltaNet: (I + L_mm)^{-1} for every diagonal block mm, one wave.  The
        // masked diagonal blocks go through LDS; then lane (g, c) solves column c of
        // block g by right-looking forward substitution with the block in registers,
        // so the 16 dependent steps wait on FMAs only.
        auto diag_inverse = [&](int b, const float* gcw) {
            if constexpr (FAM == FAM_GDN) {
                const bf16* Kb = sK(b);
                const float* G = sG(b);
                float* INV = reinterpret_cast<float*>(smem + Ly::INV_OFF);
                f32x4 acc[NTC];
#pragma unroll
                for (int mt = 0; mt < NTC; ++mt) acc[mt] = zero4();
                if constexpr (NK == 1) {
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) {
                        const bf16* kr = Kb + (16 * mt + c16) * SK + 4 * g;
                        acc[mt] = mma16(lds4(kr), lds4(kr), acc[mt]);
                        if (F32IO) {
                            acc[mt] = mma16(lds4(kr), lds4(kr + KPL), acc[mt]);
                            acc[mt] = mma16(lds4(kr + KPL), lds4(kr), acc[mt]);
                        }
                    }
                } else {
                    constexpr int NKP = NK / 2;
                    bf16x8 kv[NKP][NTC], lv[F32IO ? NKP : 1][NTC];
#pragma unroll
                    for (int kp = 0; kp < NKP; ++kp)
#pragma unroll
                        for (int mt = 0; mt < NTC; ++mt) {
                            const bf16* kr = Kb + (16 * mt + c16) * SK + 32 * kp + 8 * g;
                            kv[kp][mt] = lds8(kr);
                            if constexpr (F32IO) lv[kp][mt] = lds8(kr + KPL);
                        }
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int kp = 0; kp < NKP; ++kp)
#pragma unroll
                        for (int mt = 0; mt < NTC; ++mt) {
                            acc[mt] = mma32(kv[kp][mt], kv[kp][mt], acc[mt]);
                            if constexpr (F32IO) {
                                acc[mt] = mma32(kv[kp][mt], lv[kp][mt], acc[mt]);
                                acc[mt] = mma32(lv[kp][mt], kv[kp][mt], acc[mt]);
                            }
                        }
                }
#pragma unroll
                for (int mt = 0; mt < NTC; ++mt) {
                    const float gci = gcw[16 * mt + c16];
                    const f32x4 gt = lds4f(gcw + 16 * mt + 4 * g);
                    const f32x4 bt = lds4f(G + CH + 16 * mt + 4 * g);
                    f32x4 l;
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        l[r] = (c16 < 4 * g + r) ? bt[r] * __expf(gt[r] - gci) * acc[mt][r] : 0.f;
                    // INV block mt: LTd[i][t] = L[t][i]
                    *reinterpret_cast<f32x4*>(INV + mt * Ly::INV_BST + c16 * SLD + 4 * g) = l;
                }
                wave_lds_sync();
                if (g < NTC) {
                    const float* LTd = INV + g * Ly::INV_BST;
                    f32x4 Lc[15][4];
#pragma unroll
                    for (int m = 0; m < 15; ++m)
#pragma unroll
                        for (int q4 = (m + 1) >> 2; q4 < 4; ++q4) Lc[m][q4] = lds4f(LTd + m * SLD + 4 * q4);
                    float a[16], x[16];
#pragma unroll
                    for (int i = 0; i < 16; ++i) a[i] = 0.f;
#pragma unroll
                    for (int m = 0; m < 16; ++m) {
                        x[m] = (m == c16) ? 1.f : (m < c16 ? 0.f : -a[m]);
                        if (m < 15) {
#pragma unroll
                            for (int i = m + 1; i < 16; ++i) a[i] += Lc[m][i >> 2][i & 3] * x[m];
                        }
                    }
                    // NT[c][m] = N[m][c]: this lane's column is one contiguous NT row
                    bf16* nt_hi = sNT(b) + g * BLK + c16 * SB;
                    bf16* nt_lo = nt_hi + NTC * BLK;
#pragma unroll
                    for (int q4 = 0; q4 < 4; ++q4) {
                        const Split4 sp = split4(f32x4{x[4 * q4], x[4 * q4 + 1], x[4 * q4 + 2], x[4 * q4 + 3]});
                        *reinterpret_cast<bf16x4*>(nt_hi + 4 * q4) = sp.hi;
                        *reinterpret_cast<bf16x4*>(nt_lo + 4 * q4) = sp.lo;
                    }
                }
            }
        };

        // A-waves: state-independent blocks of chunk ci into buffer ci & 1
        auto a_work = [&](int ci) {
            const int b = ci & 1;
            float* G = sG(b);
            float* gcw = reinterpret_cast<float*>(smem + Ly::GC_OFF) + 64 * wa;
            // in-chunk cumulative log-gate, lane = token
            const float gate = lane < CH ? (FAM == FAM_GDN ? G[lane] : Ah * G[lane]) : 0.f;
            const float gc = wave_incl_scan(gate);
            const float gtot = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, gc), CH - 1));
            gcw[lane] = gc;
            if (wa == 0) {
                if (lane < CH) {
                    G[2 * CH + lane] = __expf(gc);
                    const float wt = __expf(gtot - gc);
                    G[3 * CH + lane] = (FAM == FAM_GDN) ? wt : G[lane] * wt;
                }
                if (lane < CH) G[4 * CH + lane] = gc;
                if (lane == 0) {
                    G[5 * CH] = __expf(gtot);
                    G[5 * CH + 1] = gtot;
                }
                lam_sum += gtot;
            }
            wave_lds_sync();
            if constexpr (FAM == FAM_GDN) {
                // A-wave 0 inverts the diagonal blocks; the others build the L blocks
                using NS = integral_constant<int, NA - 1>;
                switch (wa) {
                    case 0: diag_inverse(b, gcw); break;
                    case 1: items(integral_constant<int, 0>(), NS(), L_KIND(), b, gcw); break;
                    case 2: items(integral_constant<int, 1>(), NS(), L_KIND(), b, gcw); break;
                    default: items(integral_constant<int, 2>(), NS(), L_KIND(), b, gcw); break;
                }
            }
        };

        // prologue: chunk 0 staged and its blocks built; chunk 1 in flight.  While
        // the B-waves run chunk c, the A-waves commit chunk c+1 (loaded during
        // chunk c-1), issue the loads of chunk c+2, and build chunk c+1's blocks.
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
            if (ci + 1 < nch) {
                commit(ci + 1);
                if (ci + 2 < nch) prefetch(ci + 2);  // a whole chunk of lead time
            }
            __syncthreads();
            if (ci + 1 < nch) a_work(ci + 1);
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
