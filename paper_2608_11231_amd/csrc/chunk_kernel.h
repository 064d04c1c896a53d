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
// Gated DeltaNet's state waves hold S / e^lam, lam being the log decay since
// the last rescale: b_C then folds into lam, and b_t, w_t into per-token rows
// that carry e^lam (see gate_rows).
//
// The work of a chunk splits into a state-independent part (gate prefix, the
// token x token products and masks, inverses of the 16x16 diagonal blocks of
// I + L) and the state chain.  The workgroup runs them as a two-stage
// software pipeline over chunks:
//   * A-waves (NA = 4).  The stagers (3 for Gated DeltaNet, 4 for Mamba-2)
//     commit chunk c+1 from registers into LDS, form its gate prefix from
//     their own gate registers and prefetch chunk c+2 from HBM (first phase);
//     then they build chunk c+1's state-independent blocks, stored pre-split
//     (bf16 hi/lo) and transposed for direct fragment reads (second phase):
//     Gated DeltaNet's masked diagonal blocks of L (handed to the solver
//     through an LDS signal count) and strictly-lower L blocks, or Mamba-2's
//     output blocks P.  Gated DeltaNet's fourth A-wave, the solver, inverts
//     chunk c+1's diagonal blocks (second phase) and combines chunk c's
//     inverses into the off-diagonal blocks of the two 32x32 diagonal blocks
//     of (I + L)^{-1} while the B-waves start chunk c (first phase);
//   * B-waves (NB, 16*RT state rows each): chunk c's state chain -- K S^T (and
//     Gated DeltaNet's output blocks P), the two-level block substitution for
//     U (32-token halves), the outputs, the state update -- with the fp32
//     state held in MFMA accumulator registers.
// LDS holds two pipeline buffers; two workgroup barriers per chunk.  In the
// block summary the barriers order LDS traffic only (prefetched loads stay in
// flight across them); the scan keeps full barriers, which measured faster.
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
// The state waves keep S / e^lam with lam >= -LAM_FLOOR (see gate_rows): the
// stored state stays within e^32 (about 8e13) of the true one, far from fp32's range.
constexpr float LAM_FLOOR = 32.f;

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
    const int32_t* src;   // scan: when set, segment s starts from pool row src[s] of S_init
    int32_t n_src;        //   ([n_src,h_v,dv,dk]; -1 -> zero state, other ids outside -> NaN)
    int32_t init_bf16;    //   S_init holds bf16 values (widened exactly)
    void* out;            // scan: o / y [n_tok,h_v,dv] or null
    float* S_final;       // scan: final state; summary: B_out (may be null)
    float* M_out;         // summary: GDN M [n_seq,h_v,dk,dk] / SSD Lambda [n_seq,h_v], or null
    int32_t summary;      // 0: scan from S_init with outputs; 1: block summary
    int32_t tiles_b;      // row tiles over dv (state rows)
    int32_t tiles_m;      // row tiles over dk (transition rows), GDN summary only
    int32_t nb;           // B-waves per workgroup (16*nb rows per tile)
    int32_t n_units;
    int32_t wait_limit;   // polls of the solver's bounded wait for the stagers' signals
    // Mamba-2 scan kernel only: with pieces > 1 every segment is cut into that
    // many pieces of whole chunks (the sequence-parallel scan's cut), piece 0
    // starting from the segment's initial state and the others from zero;
    // every piece's end state and log-decay sum go to piece_B / piece_L
    // ([n_seq * pieces, h_v, dv, dk] / [n_seq * pieces, h_v]) instead of S_final
    int32_t pieces;
    float* piece_B;
    float* piece_L;
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
    // gate rows: raw gate | beta | b e^lam | w e^-lam' | cumulative gate gc |
    // state factor, e^lam' (4) | beta b e^lam   (lam / lam': the stored state's
    // log scale before / after the chunk; Mamba-2: lam = lam' = 0)
    static constexpr int BB_ROW = 5 * CH + 4;
    static constexpr size_t G_SZ = al((6 * CH + 4) * 4);
    static constexpr size_t LT_SZ = HAS_L ? al(size_t(NOFF) * BLK * 2 * 2) : 0;
    static constexpr size_t NT_SZ = HAS_L ? al(size_t(NTC) * BLK * 2 * 2) : 0;
    static constexpr size_t PT_SZ = HAS_Q ? al(size_t(NPB) * BLK * PL * 2) : 0;
    // off-diagonal blocks T_10, T_32 of the two 32x32 diagonal blocks of (I + L)^{-1}, hi / lo
    static constexpr size_t TT_SZ = (HAS_L && NTC == 4) ? al(size_t(2) * BLK * 2 * 2) : 0;
    static constexpr size_t K_OFF = 0;
    static constexpr size_t Q_OFF = K_OFF + K_SZ;
    static constexpr size_t V_OFF = Q_OFF + Q_SZ;
    static constexpr size_t G_OFF = V_OFF + V_SZ;
    static constexpr size_t LT_OFF = G_OFF + G_SZ;
    static constexpr size_t NT_OFF = LT_OFF + LT_SZ;
    static constexpr size_t PT_OFF = NT_OFF + NT_SZ;
    static constexpr size_t TT_OFF = PT_OFF + PT_SZ;
    static constexpr size_t BUF = TT_OFF + TT_SZ;  // one pipeline buffer
    static constexpr size_t GC_OFF = 2 * BUF;      // per A-wave gate prefix
    static constexpr size_t INV_OFF = GC_OFF + al(NA * 64 * 4);
    static constexpr int INV_BST = 16 * SLD + 4;      // f32 stride of inverse scratch blocks (bank shift)
    // count of stager signals "this chunk's masked diagonal blocks are in LDS"
    static constexpr size_t CNT_OFF = INV_OFF + (HAS_L ? al(size_t(NTC) * INV_BST * 4) : 0);
    static constexpr size_t BYTES = CNT_OFF + (HAS_L ? 16 : 0);
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

template <int FAM, int DK, int CH, bool F32IO, int NB, bool SUMMARY, int RT = 1>
__global__ __launch_bounds__(64 * (NB + NA), (NB + NA) / 4) void chunk_kernel(ScanArgs p) {
    static_assert(RT == 1 || SUMMARY, "several row tiles per wave: block summaries only");
    using Ly = ChunkLds<FAM, DK, CH, F32IO, NB * RT, SUMMARY>;
    constexpr int NTC = CH / 16, NTK = DK / 16;
    constexpr int SK = Ly::SK, SV = Ly::SV, SB = Ly::SB, BLK = Ly::BLK, SLD = Ly::SLD;
    constexpr int NOFF = Ly::NOFF, NPB = Ly::NPB;
    constexpr int KPL = CH * SK, VPL = CH * SV;  // lo-plane offsets (fp32 io)
    extern __shared__ __align__(16) char smem[];

    const int tid = threadIdx.x;
    // wave index as a scalar: role and slot branches below are then uniform
    // scalar branches instead of exec-masked divergent regions
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63, g = lane >> 4, c16 = lane & 15;
    auto chunk_barrier = []() {
        if constexpr (SUMMARY) lds_barrier();
        else __syncthreads();
    };
    const bool is_b = w < NB;
    const int wa = w - NB;            // A-wave index
    const int tid_a = tid - 64 * NB;  // thread index among the A-waves
    if constexpr (FAM == FAM_GDN) {
        // stager -> solver signal count (ordered before its first use by the prologue barrier)
        if (tid == 0) *reinterpret_cast<uint32_t*>(smem + Ly::CNT_OFF) = 0u;
    }

    // ---- work unit.  Order of the units, innermost first: the row tiles and the
    // value heads of one q/k head (they read the same token rows, so they share
    // an L2), then hpx = h_qk / 8 adjacent q/k heads (neighbouring row segments
    // of the same tokens, read at the same time), then the segment, then the
    // group of hpx q/k heads.  xcd_unit hands each XCD a contiguous range, i.e.
    // one head group of every segment: ragged segment lengths then load the
    // XCDs evenly (giving each XCD whole segments left the fold 13% unbalanced
    // at 32K and the ragged batch 50%).
    const int tiles = p.tiles_b + p.tiles_m;
    const int hr = p.h_v / p.h_qk;  // value heads per q/k head
    const int hpx = (p.h_qk % 8 == 0) ? p.h_qk / 8 : 1;
    const int u = xcd_unit(blockIdx.x, p.n_units);
    const int inner = u % (tiles * hr), outer = u / (tiles * hr);
    const int tile = inner % tiles;
    const int hsub = outer % hpx, o2 = outer / hpx;
    const int s = o2 % p.n_seq;
    const int hq = (o2 / p.n_seq) * hpx + hsub;
    const int h = hq * hr + inner / tiles;
    const bool mtile = tile >= p.tiles_b;
    const int row0 = (mtile ? tile - p.tiles_b : tile) * 16 * NB * RT;  // first state row of the tile
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
    auto sTT = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::TT_OFF); };

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
            // more than five blocks (one or two state waves building all of a
            // chunk's output blocks) are built in batches of four; with fp32 io
            // (fragments with lo planes) in batches of two, or one by one for a
            // single state wave: one batch's fragments, double-buffered, then fit
            // the registers with the state
            constexpr int BAT = F32IO ? (NMY > 5 ? 1 : (NMY > 3 ? 2 : NMY)) : (NMY > 5 ? 4 : NMY);
            constexpr int NBAT = (NMY + BAT - 1) / BAT;
            auto batch = [&](auto bi_c) {
                constexpr int I0 = decltype(bi_c)::value * BAT;
                constexpr int BN = (NMY - I0) < BAT ? (NMY - I0) : BAT;
                auto item_mt = [](int i) {
                    return KL ? off_mt(SLOT + (I0 + i) * NSLOT) : low_mt(SLOT + (I0 + i) * NSLOT);
                };
                auto item_nt = [](int i) {
                    const int j = SLOT + (I0 + i) * NSLOT;
                    return KL ? j - off_index(off_mt(j), 0) : j - low_index(low_mt(j), 0);
                };
                f32x4 acc[BN];
#pragma unroll
                for (int i = 0; i < BN; ++i) acc[i] = zero4();
                if constexpr (NK == 1) {
#pragma unroll
                    for (int i = 0; i < BN; ++i) {
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
                    bf16x8 fa[2][FPL][BN], fb[2][FPL][BN];
                    auto fetch = [&](int kp, int buf) {
#pragma unroll
                        for (int i = 0; i < BN; ++i) {
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
                        for (int i = 0; i < BN; ++i) {
                            acc[i] = mma32(fa[cb][0][i], fb[cb][0][i], acc[i]);
                            if constexpr (F32IO) {
                                acc[i] = mma32(fa[cb][0][i], fb[cb][FPL - 1][i], acc[i]);
                                acc[i] = mma32(fa[cb][FPL - 1][i], fb[cb][0][i], acc[i]);
                            }
                        }
                    }
                }
#pragma unroll
                for (int i = 0; i < BN; ++i) {
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
            };
            static_for<0, NBAT>(batch);
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
        // ---- the state: RT row tiles per wave, tile rt covering rows row_of(rt);
        // acc layout: S[rt][nt] holds S[row][16nt + 4g + r]
        auto row_of = [&](int rt) { return row0 + 16 * (RT * w + rt) + c16; };
        const bf16x8 negI = neg_eye(g, c16);  // hi / lo splits on the matrix core
        const bf16x8 negIh = neg_eye_hi(g, c16);
        f32x4 S[RT][NTK];
        // initial state row: segment s's own (S_init) or, with src, a pool row
        // (LinearKV's single cached state read straight from the cache pool)
        int64_t init_row = s;
        float init_fill = 0.f;
        bool init_load = !SUMMARY && p.S_init;
        if (!SUMMARY && p.src) {
            const int32_t id = p.src[s];
            init_row = id;
            if (id < 0 || id >= p.n_src) {
                init_load = false;
                init_fill = id == -1 ? 0.f : __builtin_nanf("");
            }
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int nt = 0; nt < NTK; ++nt) {
                const int row = row_of(rt);
                const int64_t e = ((init_row * p.h_v + h) * p.dv + row) * DK + 16 * nt + 4 * g;
                if (init_load && p.init_bf16) {
                    const uint2 u = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(p.S_init) + e);
                    S[rt][nt] = f32x4{__builtin_bit_cast(float, u.x << 16), __builtin_bit_cast(float, u.x & 0xffff0000u),
                                      __builtin_bit_cast(float, u.y << 16), __builtin_bit_cast(float, u.y & 0xffff0000u)};
                } else if (init_load) {
                    S[rt][nt] = *reinterpret_cast<const f32x4*>(p.S_init + e);
                } else if (!SUMMARY && p.src) {
                    S[rt][nt] = f32x4{init_fill, init_fill, init_fill, init_fill};
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r) S[rt][nt][r] = (mtile && row == 16 * nt + 4 * g + r) ? 1.f : 0.f;
                }
            }
        // bf16 hi / lo parts of the state, refreshed after every state update
        bf16x4 Sh[RT][NTK], Sl[RT][NTK];
        auto split_state = [&]() {
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                // 64-token chunks: S comes from a 32-wide MFMA chain, which the
                // 32-wide split product may follow (dk tiles in pairs, as K S^T
                // reads them); 16-token chunks update S 16-wide, and one chain
                // never mixes the two shapes
                if constexpr (NTC == 4 && NTK % 2 == 0) {
#pragma unroll
                    for (int nt = 0; nt < NTK; nt += 2) {
                        const Split8 sp = split8_mm(S[rt][nt], S[rt][nt + 1], negI, negIh);
                        Sh[rt][nt] = sp.hi0;
                        Sh[rt][nt + 1] = sp.hi1;
                        Sl[rt][nt] = sp.lo0;
                        Sl[rt][nt + 1] = sp.lo1;
                    }
                } else {
#pragma unroll
                    for (int nt = 0; nt < NTK; ++nt) {
                        const Split4 sp = NTC == 4 ? split4_mm(S[rt][nt], negI) : split4(S[rt][nt]);
                        Sh[rt][nt] = sp.hi;
                        Sl[rt][nt] = sp.lo;
                    }
                }
            }
        };
        split_state();
        chunk_barrier();  // prologue: chunk 0 staged by the A-waves
        for (int ci = 0; ci < nch; ++ci) {
            const int b = ci & 1;
            const int64_t c0 = t0 + (int64_t)ci * CH;
            const int n = (int)((t1 - c0) < CH ? (t1 - c0) : CH);
            chunk_barrier();
            // ================= phase I: K S^T and the delta-rule right-hand side
            // X: v of the chunk (state rows), later the substitution's right-hand
            // side.  The scan and Mamba-2 read v here, ahead of K S^T; a Gated
            // DeltaNet block summary reads it where it is combined (below), so its
            // transition rows carry no value of X across the branch
            constexpr bool V_EARLY = !SUMMARY || FAM == FAM_SSD;
            f32x4 X[RT][NTC];
            {
                const bf16* Kb = sK(b);
                const float* G = sG(b);
                if (V_EARLY && load_v) {
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                        for (int mt = 0; mt < NTC; ++mt) {
                            const int col = 16 * (RT * w + rt);
                            X[rt][mt] = to_f32(lds4_tr(sV(b), SV, 16 * mt, col, g, c16));
                            if (F32IO) X[rt][mt] += to_f32(lds4_tr(sV(b) + VPL, SV, 16 * mt, col, g, c16));
                        }
                }
                if (FAM == FAM_GDN && with_out) {
                    // Gated DeltaNet: this chunk's output blocks P, shared by the B-waves
                    // (read after the barrier).  The stagers' second phase is full with
                    // the L blocks; Mamba-2's stagers build P instead.
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
                    // K S^T for all token tiles at once (interleaved chains, passes pass-major)
                    f32x4 ks[RT][NTC];
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                        for (int mt = 0; mt < NTC; ++mt) ks[rt][mt] = zero4();
                    if constexpr (RT == 1)
                        mgemm_rows<NTC, F32IO, true>(Kb + c16 * SK, 16 * SK, KPL, Sh[0], Sl[0], NTK, g, ks[0]);
                    else
                        mgemm_rows_rt<NTC, RT, NTK, F32IO, true>(Kb + c16 * SK, 16 * SK, KPL, Sh, Sl, g, ks);
                    // X = beta (v - b k S^T) = beta v - (beta b) k S^T  (v = 0 on transition tiles)
                    if (load_v) {
#pragma unroll
                        for (int mt = 0; mt < NTC; ++mt) {
                            const f32x4 bb = lds4f(G + Ly::BB_ROW + 16 * mt + 4 * g);
                            const f32x4 be = lds4f(G + CH + 16 * mt + 4 * g);
#pragma unroll
                            for (int rt = 0; rt < RT; ++rt) {
                                if constexpr (!V_EARLY) {
                                    const int col = 16 * (RT * w + rt);
                                    X[rt][mt] = to_f32(lds4_tr(sV(b), SV, 16 * mt, col, g, c16));
                                    if (F32IO) X[rt][mt] += to_f32(lds4_tr(sV(b) + VPL, SV, 16 * mt, col, g, c16));
                                }
#pragma unroll
                                for (int r = 0; r < 4; ++r)
                                    X[rt][mt][r] = be[r] * X[rt][mt][r] - bb[r] * ks[rt][mt][r];
                            }
                        }
                    } else {
#pragma unroll
                        for (int mt = 0; mt < NTC; ++mt) {
                            const f32x4 bb = lds4f(G + Ly::BB_ROW + 16 * mt + 4 * g);
#pragma unroll
                            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                                for (int r = 0; r < 4; ++r) X[rt][mt][r] = -bb[r] * ks[rt][mt][r];
                        }
                    }
                }
            }
            // Outputs (RT == 1 only) are formed transposed, O^T = S Q^T + U^T P^T:
            // tile mt holds O[16mt + c16][this wave's rows 4g..4g+3], so each lane
            // stores 4 consecutive state rows of one token.  S Q^T does not depend
            // on U: it is formed here, while the B-waves would otherwise wait for
            // the A-waves at the barrier.
            f32x4 OT[NTC];
            if (with_out) {
                const bf16* Qb = sQ(b);
#pragma unroll
                for (int mt = 0; mt < NTC; ++mt) OT[mt] = zero4();
                if constexpr (NTK == 1) {
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) {
                        const bf16* qr = Qb + (16 * mt + c16) * SK + 4 * g;
                        OT[mt] = mma16(Sh[0][0], lds4(qr), OT[mt]);
                        if (F32IO) {
                            OT[mt] = mma16(Sl[0][0], lds4(qr), OT[mt]);
                            OT[mt] = mma16(Sh[0][0], lds4(qr + KPL), OT[mt]);
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
                            OT[mt] = mma32(Sh[0][2 * kp], Sh[0][2 * kp + 1], qh[kp][mt], OT[mt]);
                            if constexpr (F32IO) {
                                OT[mt] = mma32(Sl[0][2 * kp], Sl[0][2 * kp + 1], qh[kp][mt], OT[mt]);
                                OT[mt] = mma32(Sh[0][2 * kp], Sh[0][2 * kp + 1], ql[kp][mt], OT[mt]);
                            }
                        }
                }
            }
            chunk_barrier();
            // ================= phase II: substitution, outputs, state update
            {
                const bf16* Kb = sK(b);
                const float* G = sG(b);
                f32x4 U[RT][NTC];
                bf16x4 Uh[RT][NTC], Ul[RT][NTC];
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
                    // U = (I + L)^{-1} X over 32-token halves A = blocks {0, 1}, B = {2, 3}:
                    //   U_A = T_A X_A,  U_B = T_B (X_B - L_BA U_A),
                    // with T_A = [[N_0, 0], [T_10, N_1]], T_B = [[N_2, 0], [T_32, N_3]] (the
                    // 16x16 diagonal inverses N and T_10 = -N_1 L_10 N_0, T_32 = -N_3 L_32 N_2
                    // come from the A-waves).  Three dependent stages, the row tiles
                    // interleaved; each product's three passes chain on one accumulator
                    // (the row tiles and output tiles of a stage keep RT * 2 chains in flight).
                    // All fragments are requested before the first product.
                    const bf16* LT = sLT(b);
                    const bf16* NT = sNT(b);
                    bf16x4 Nh[NTC], Nl[NTC];
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) {
                        Nh[mt] = lds4_tr(NT + mt * BLK, SB, 0, 0, g, c16);
                        Nl[mt] = lds4_tr(NT + (NTC + mt) * BLK, SB, 0, 0, g, c16);
                    }
                    auto split_u = [&](int rt, int mt, f32x4 v) {
                        U[rt][mt] = v;
                        const Split4 us = split4_mm(v, negI);
                        Uh[rt][mt] = us.hi;
                        Ul[rt][mt] = us.lo;
                    };
                    // token tiles mt, mt + 1 together (the 32-wide slice later products read)
                    auto split_u2 = [&](int rt, int mt, f32x4 v0, f32x4 v1) {
                        U[rt][mt] = v0;
                        U[rt][mt + 1] = v1;
                        const Split8 us = split8_mm(v0, v1, negI, negIh);
                        Uh[rt][mt] = us.hi0;
                        Uh[rt][mt + 1] = us.hi1;
                        Ul[rt][mt] = us.lo0;
                        Ul[rt][mt + 1] = us.lo1;
                    };
                    if constexpr (NTC == 1) {
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt) {
                            const Split4 xs = split4_mm(X[rt][0], negI);
                            const f32x4 u0 = mma16(Nh[0], xs.hi, zero4());
                            f32x4 u1 = mma16(Nh[0], xs.lo, zero4());
                            u1 = mma16(Nl[0], xs.hi, u1);
                            split_u(rt, 0, u0 + u1);
                        }
                    } else {
                        static_assert(NTC == 4, "chunk of 16 or 64 tokens");
                        const bf16* TT = sTT(b);
                        const bf16x4 t10h = lds4_tr(TT, SB, 0, 0, g, c16);
                        const bf16x4 t32h = lds4_tr(TT + BLK, SB, 0, 0, g, c16);
                        const bf16x4 t10l = lds4_tr(TT + 2 * BLK, SB, 0, 0, g, c16);
                        const bf16x4 t32l = lds4_tr(TT + 3 * BLK, SB, 0, 0, g, c16);
                        // -L_20, -L_21, -L_30, -L_31 (strictly-lower blocks 1..4), hi / lo
                        bf16x4 Lh[4], Ll[4];
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            Lh[j] = lds4_tr(LT + (1 + j) * BLK, SB, 0, 0, g, c16);
                            Ll[j] = lds4_tr(LT + (NOFF + 1 + j) * BLK, SB, 0, 0, g, c16);
                        }
                        // stage 1: U_0 = N_0 X_0, U_1 = T_10 X_0 + N_1 X_1
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt) {
                            const Split8 x01 = split8_mm(X[rt][0], X[rt][1], negI, negIh);
                            f32x4 u0 = mma16(Nh[0], x01.hi0, zero4());
                            f32x4 u1 = mma32(t10h, Nh[1], x01.hi0, x01.hi1, zero4());
                            u0 = mma16(Nh[0], x01.lo0, u0);
                            u1 = mma32(t10h, Nh[1], x01.lo0, x01.lo1, u1);
                            u0 = mma16(Nl[0], x01.hi0, u0);
                            u1 = mma32(t10l, Nl[1], x01.hi0, x01.hi1, u1);
                            split_u2(rt, 0, u0, u1);
                        }
                        // stage 2: R_2 = X_2 - L_20 U_0 - L_21 U_1, R_3 = X_3 - L_30 U_0 - L_31 U_1
                        Split8 x23[RT];
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt) {
                            f32x4 r2 = mma32(Lh[0], Lh[1], Uh[rt][0], Uh[rt][1], X[rt][2]);
                            f32x4 r3 = mma32(Lh[2], Lh[3], Uh[rt][0], Uh[rt][1], X[rt][3]);
                            r2 = mma32(Lh[0], Lh[1], Ul[rt][0], Ul[rt][1], r2);
                            r3 = mma32(Lh[2], Lh[3], Ul[rt][0], Ul[rt][1], r3);
                            r2 = mma32(Ll[0], Ll[1], Uh[rt][0], Uh[rt][1], r2);
                            r3 = mma32(Ll[2], Ll[3], Uh[rt][0], Uh[rt][1], r3);
                            x23[rt] = split8_mm(r2, r3, negI, negIh);
                        }
                        // stage 3: U_2 = N_2 R_2, U_3 = T_32 R_2 + N_3 R_3
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt) {
                            f32x4 u2 = mma16(Nh[2], x23[rt].hi0, zero4());
                            f32x4 u3 = mma32(t32h, Nh[3], x23[rt].hi0, x23[rt].hi1, zero4());
                            u2 = mma16(Nh[2], x23[rt].lo0, u2);
                            u3 = mma32(t32h, Nh[3], x23[rt].lo0, x23[rt].lo1, u3);
                            u2 = mma16(Nl[2], x23[rt].hi0, u2);
                            u3 = mma32(t32l, Nl[3], x23[rt].hi0, x23[rt].hi1, u3);
                            split_u2(rt, 2, u2, u3);
                        }
                    }
                } else {
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                        for (int mt = 0; mt < NTC; ++mt) {
                            const int col = 16 * (RT * w + rt);
                            U[rt][mt] = X[rt][mt];
                            Uh[rt][mt] = lds4_tr(sV(b), SV, 16 * mt, col, g, c16);
                            Ul[rt][mt] = F32IO ? lds4_tr(sV(b) + VPL, SV, 16 * mt, col, g, c16) : zero_bf16x4();
                        }
                }
                if (with_out) {
                    const float coef = (FAM == FAM_GDN) ? p.scale : 1.f;
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) OT[mt] *= coef * G[2 * CH + 16 * mt + c16];
                    // + U^T P^T: tile mt contracts over token blocks 0..mt, pairs of blocks per MFMA
                    if constexpr (NTC == 1) {
                        const bf16x4 x = Pf[0][0];
                        OT[0] = mma16(Uh[0][0], x, OT[0]);
                        if (F32IO) {
                            OT[0] = mma16(Ul[0][0], x, OT[0]);
                            OT[0] = mma16(Uh[0][0], Pf[PPL - 1][0], OT[0]);
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
                                const bf16x4 u1h = two ? Uh[0][kp + 1] : zero_bf16x4();
                                OT[mt] = mma32(Uh[0][kp], u1h, x0, x1, OT[mt]);
                                if (F32IO) {
                                    const bf16x4 u1l = two ? Ul[0][kp + 1] : zero_bf16x4();
                                    OT[mt] = mma32(Ul[0][kp], u1l, x0, x1, OT[mt]);
                                    const bf16x4 y0 = Pf[PPL - 1][j0];
                                    const bf16x4 y1 = two ? Pf[PPL - 1][j0 + 1] : zero_bf16x4();
                                    OT[mt] = mma32(Uh[0][kp], u1h, y0, y1, OT[mt]);
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
                // S <- rho S + K^T diag(w) U   (rho: 1, or the rescale of gate_rows;
                // all dk tiles and row tiles interleaved)
                bf16x4 Wh[RT][NTC], Wl[RT][NTC];
                if constexpr (NTC == 4) {
#pragma unroll
                    for (int mt = 0; mt < NTC; mt += 2) {
                        const f32x4 w0 = lds4f(G + 3 * CH + 16 * mt + 4 * g);
                        const f32x4 w1 = lds4f(G + 3 * CH + 16 * mt + 16 + 4 * g);
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt) {
                            const Split8 sp = split8_mm(w0 * U[rt][mt], w1 * U[rt][mt + 1], negI, negIh);
                            Wh[rt][mt] = sp.hi0;
                            Wh[rt][mt + 1] = sp.hi1;
                            Wl[rt][mt] = sp.lo0;
                            Wl[rt][mt + 1] = sp.lo1;
                        }
                    }
                } else {
#pragma unroll
                    for (int mt = 0; mt < NTC; ++mt) {
                        const f32x4 wt = lds4f(G + 3 * CH + 16 * mt + 4 * g);
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt) {
                            const Split4 sp = split4_mm(wt * U[rt][mt], negI);
                            Wh[rt][mt] = sp.hi;
                            Wl[rt][mt] = sp.lo;
                        }
                    }
                }
                // state factor: 1 (the decay stays in the stored scale) or a rescale;
                // compared as bits so the branch is scalar
                const uint32_t rho = (uint32_t)__builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, G[5 * CH]));
                if (rho != 0x3f800000u) {
                    const float r = __builtin_bit_cast(float, rho);
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                        for (int nt = 0; nt < NTK; ++nt) S[rt][nt] = r * S[rt][nt];
                }
                if constexpr (RT == 1)
                    mgemm_tr<DK, NTK, F32IO, true>(Kb, KPL, SK, Wh[0], Wl[0], NTC, g, c16, S[0]);
                else
                    mgemm_tr_rt<DK, NTK, RT, NTC, F32IO, true>(Kb, KPL, SK, Wh, Wl, g, c16, S);
                split_state();  // for the next chunk, ahead of its barrier
            }
        }
        float* dst = mtile ? p.M_out : p.S_final;
        if (dst) {
            // back from the stored scale (the last chunk's gate rows are still in place)
            if (nch > 0) {
                const float sc = sG((nch - 1) & 1)[5 * CH + 1];
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                    for (int nt = 0; nt < NTK; ++nt) S[rt][nt] = sc * S[rt][nt];
            }
            const int rows = mtile ? DK : p.dv;
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int nt = 0; nt < NTK; ++nt)
                    *reinterpret_cast<f32x4*>(dst + ((int64_t(s) * p.h_v + h) * rows + row_of(rt)) * DK + 16 * nt +
                                              4 * g) = S[rt][nt];
        }
    } else {
        // ---- A-waves: HBM -> register prefetch and register -> LDS commit of a chunk
        // Gated DeltaNet: A-waves 0..NA-2 stage tiles and build the L blocks; A-wave
        // NA-1 (the solver) builds the triangular inverses.
        constexpr int NSTG = (FAM == FAM_GDN) ? NA - 1 : NA;
        const bool stager = wa < NSTG;
        KQTile<CH, DK, F32IO, 64 * NSTG> pk, pq;
        TileRegs<CH, 16 * NB * RT, F32IO, 64 * NSTG> pv;
        uint32_t pg = 0u, pb = 0u;  // gates stay raw bits until commit (no early wait on the loads)
        float lam_sum = 0.f;
        float lam = 0.f;  // stager 0: log scale of the state waves' stored state
        constexpr int ES = F32IO ? 4 : 2;
        const uint32_t qk_rb = (uint32_t)(p.h_qk * DK * ES), v_rb = (uint32_t)(p.h_v * p.dv * ES);
        // Chunk loads go through buffer resources that end at the chunk's last
        // valid row: rows past the segment's end (and lanes past the tile) read
        // as zero by the hardware range check, so the loads need no branches
        // and the per-lane offsets are the same for every chunk.
        const uint32_t gbytes = (FAM == FAM_GDN && p.gate_bf16) ? 2u : 4u;
        // Gated DeltaNet: the stagers' own work on a chunk (its L blocks and
        // diagonal blocks) reads only k and the gates, so q and v are committed
        // in the other half of the chunk, next to that work: the half before it
        // (commit, prefetch) is otherwise longer than the state waves' phase I.
        // Mamba-2 builds its output blocks from q there, so it commits q first.
        constexpr bool QV_LATE = FAM == FAM_GDN;
        auto prefetch_qv = [&](int ci) {
            const int64_t c0 = t0 + (int64_t)ci * CH;
            const uint32_t n = (uint32_t)((t1 - c0) < CH ? (t1 - c0) : CH);
            const int64_t qk_off = (c0 * p.h_qk + hq) * (int64_t)DK * ES;
            if (with_out)
                pq.load_buf(make_rsrc(reinterpret_cast<const char*>(p.q) + qk_off, n * qk_rb), 0u, qk_rb, tid_a);
            if (load_v)
                pv.load_buf(make_rsrc(reinterpret_cast<const char*>(p.v) +
                                          ((c0 * p.h_v + h) * (int64_t)p.dv + row0) * ES,
                                      n * v_rb),
                            0u, v_rb, tid_a);
        };
        auto commit_qv = [&](int ci) {
            const int b = ci & 1;
            if (with_out) pq.commit(sQ(b), SK, KPL, tid_a);
            if (load_v) pv.commit(sV(b), SV, VPL, tid_a);
        };
        auto prefetch = [&](int ci) {
            const int64_t c0 = t0 + (int64_t)ci * CH;
            const uint32_t n = (uint32_t)((t1 - c0) < CH ? (t1 - c0) : CH);
            const int64_t qk_off = (c0 * p.h_qk + hq) * (int64_t)DK * ES;
            pk.load_buf(make_rsrc(reinterpret_cast<const char*>(p.k) + qk_off, n * qk_rb), 0u, qk_rb, tid_a);
            if (!QV_LATE) prefetch_qv(ci);
            // gates: lane t < CH of every stager takes token t of the chunk (raw
            // bits, widened at commit; each stager forms the gate prefix itself)
            const int64_t g_off = (c0 * p.h_v + h) * (int64_t)gbytes;
            const uint32_t g_rb = (uint32_t)p.h_v * gbytes;
            const uint32_t goff = lane < CH ? (uint32_t)lane * g_rb : 0xffffffffu;
            const __amdgpu_buffer_rsrc_t rg = make_rsrc(reinterpret_cast<const char*>(p.g) + g_off, n * g_rb);
            if (FAM == FAM_GDN) {
                const __amdgpu_buffer_rsrc_t rb = make_rsrc(reinterpret_cast<const char*>(p.beta) + g_off, n * g_rb);
                if (p.gate_bf16) {
                    pg = buf_load2(rg, goff);
                    pb = buf_load2(rb, goff);
                } else {
                    pg = buf_load4(rg, goff);
                    pb = buf_load4(rb, goff);
                }
            } else {
                pg = buf_load4(rg, goff);  // dt
            }
        };
        auto commit = [&](int ci) {
            const int b = ci & 1;
            pk.commit(sK(b), SK, KPL, tid_a);
            if (!QV_LATE) commit_qv(ci);
            if (tid_a < CH) {
                float* G = sG(b);
                const bool b16 = FAM == FAM_GDN && p.gate_bf16;
                G[tid_a] = __builtin_bit_cast(float, b16 ? pg << 16 : pg);
                G[CH + tid_a] = __builtin_bit_cast(float, b16 ? pb << 16 : pb);
            }
        };
        // Per-chunk gate rows from this stager's own gate registers (run right
        // after commit, before the next prefetch reuses them): the in-chunk
        // cumulative log-gate in the wave's private row gcw (lane = token), and,
        // from stager 0, the rows b, w, gc, beta b and the state factors that the
        // B-waves read.
        auto gate_rows = [&](int ci) {
            const int b = ci & 1;
            float* G = sG(b);
            float* gcw = reinterpret_cast<float*>(smem + Ly::GC_OFF) + 64 * wa;
            const bool b16 = FAM == FAM_GDN && p.gate_bf16;
            const float graw = __builtin_bit_cast(float, b16 ? pg << 16 : pg);
            const float gate = lane < CH ? (FAM == FAM_GDN ? graw : Ah * graw) : 0.f;
            const float gc = wave_incl_scan(gate);
            const float gtot = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, gc), CH - 1));
            gcw[lane] = gc;
            if (wa == 0) {
                // The state waves hold S / e^lam (lam = the log decay since the last
                // rescale), so the chunk's decay b_C needs no pass over the state:
                // it moves into lam, and the per-token rows carry e^lam instead.
                // Once lam would drop below -LAM_FLOOR the state is rescaled by
                // e^lam (the state factor below) and lam restarts at 0, which keeps
                // S / e^lam within e^LAM_FLOOR of S.  Mamba-2 rescales every chunk
                // (lam stays 0: the plain b_C S form, which its eight-wave scan
                // kernel reproduces bit for bit).
                const float lam_in = lam;
                float lam_out = lam_in + gtot, rho = 1.f;
                if (FAM != FAM_GDN || lam_out < -LAM_FLOOR) {
                    rho = __expf(lam_out);
                    lam_out = 0.f;
                }
                if (lane < CH) {
                    const float bt = __expf(gc + lam_in);  // b_t against the stored state
                    G[2 * CH + lane] = bt;
                    const float wt = __expf(gtot - gc - lam_out);
                    G[3 * CH + lane] = (FAM == FAM_GDN) ? wt : graw * wt;
                    G[4 * CH + lane] = gc;
                    if (FAM == FAM_GDN) G[Ly::BB_ROW + lane] = __builtin_bit_cast(float, b16 ? pb << 16 : pb) * bt;
                }
                if (lane == 0) {
                    G[5 * CH] = rho;                    // state factor of this chunk's update
                    G[5 * CH + 1] = __expf(lam_out);    // stored -> true state after it
                }
                lam = lam_out;
                lam_sum += gtot;
            }
        };

        // Gated DeltaNet: (I + L_mm)^{-1} of the diagonal blocks.  The stagers put
        // the masked diagonal blocks in LDS (diag_prep; stager a takes blocks
        // NSTG-1-a, 2 NSTG-1-a, ...) and signal the solver through an LDS counter;
        // the solver inverts them all at once by right-looking forward substitution
        // with each block in registers, so the 16 dependent steps wait on FMAs only.
        // A stager's blocks are formed together: every fragment and gate is
        // requested first, then the blocks run as independent accumulation chains.
        auto diag_prep = [&](auto first_c, int b, const float* gcw) {
            constexpr int F = decltype(first_c)::value;
            constexpr int NMY = F < NTC ? (NTC - F + NSTG - 1) / NSTG : 0;
            if constexpr (FAM == FAM_GDN && NMY > 0) {
                const float* G = sG(b);
                auto krow = [&](int i) { return sK(b) + (16 * (F + i * NSTG) + c16) * SK; };
                f32x4 acc[NMY], gt[NMY], bt[NMY];
                float gci[NMY];
#pragma unroll
                for (int i = 0; i < NMY; ++i) acc[i] = zero4();
                auto gates = [&]() {
#pragma unroll
                    for (int i = 0; i < NMY; ++i) {
                        const int mt = F + i * NSTG;
                        gci[i] = gcw[16 * mt + c16];
                        gt[i] = lds4f(gcw + 16 * mt + 4 * g);
                        bt[i] = lds4f(G + CH + 16 * mt + 4 * g);
                    }
                };
                if constexpr (NK == 1) {
#pragma unroll
                    for (int i = 0; i < NMY; ++i) {
                        const bf16* kr = krow(i);
                        acc[i] = mma16(lds4(kr + 4 * g), lds4(kr + 4 * g), acc[i]);
                        if (F32IO) {
                            acc[i] = mma16(lds4(kr + 4 * g), lds4(kr + KPL + 4 * g), acc[i]);
                            acc[i] = mma16(lds4(kr + KPL + 4 * g), lds4(kr + 4 * g), acc[i]);
                        }
                    }
                    gates();
                } else {
                    constexpr int NKP = NK / 2;
                    bf16x8 kv[NKP][NMY], lv[F32IO ? NKP : 1][NMY];
#pragma unroll
                    for (int kp = 0; kp < NKP; ++kp)
#pragma unroll
                        for (int i = 0; i < NMY; ++i) {
                            kv[kp][i] = lds8(krow(i) + 32 * kp + 8 * g);
                            if constexpr (F32IO) lv[kp][i] = lds8(krow(i) + KPL + 32 * kp + 8 * g);
                        }
                    gates();
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int kp = 0; kp < NKP; ++kp)
#pragma unroll
                        for (int i = 0; i < NMY; ++i) {
                            acc[i] = mma32(kv[kp][i], kv[kp][i], acc[i]);
                            if constexpr (F32IO) {
                                acc[i] = mma32(kv[kp][i], lv[kp][i], acc[i]);
                                acc[i] = mma32(lv[kp][i], kv[kp][i], acc[i]);
                            }
                        }
                }
#pragma unroll
                for (int i = 0; i < NMY; ++i) {
                    float* INV = reinterpret_cast<float*>(smem + Ly::INV_OFF) + (F + i * NSTG) * Ly::INV_BST;
                    f32x4 l;
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        l[r] = (c16 < 4 * g + r) ? bt[i][r] * __expf(gt[i][r] - gci[i]) * acc[i][r] : 0.f;
                    // LTd[i][t] = L[t][i]
                    *reinterpret_cast<f32x4*>(INV + c16 * SLD + 4 * g) = l;
                }
            }
        };
        uint32_t* diag_cnt = reinterpret_cast<uint32_t*>(smem + Ly::CNT_OFF);
        // One wave inverts every diagonal block: lane c of lane group g solves
        // column c of block g (the masked blocks were left in LDS by diag_prep).
        // A wait that gave up (ok false) stores NaN blocks: the chunk's state and
        // outputs then become NaN instead of values built from stale LDS.
        auto diag_solve_all = [&](int b, bool ok) {
            if constexpr (FAM == FAM_GDN) {
                if (g < NTC) {
                    const float* LTd = reinterpret_cast<const float*>(smem + Ly::INV_OFF) + g * Ly::INV_BST;
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
                    if (!ok) {
#pragma unroll
                        for (int m = 0; m < 16; ++m) x[m] = __builtin_nanf("");
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
                    asm volatile("" ::: "memory");  // keep the stores in this branch
                }
                wave_lds_sync();  // N is read back by t_blocks
            }
        };

        // Gated DeltaNet, 64-token chunks: T_10 = -N_1 L_10 N_0 and T_32 = -N_3 L_32 N_2,
        // the off-diagonal blocks of the 32x32 diagonal blocks of (I + L)^{-1}, from the
        // stored -L and N blocks of buffer b.  Y = (-L)^T N_i^T = -(N_i L)^T, whose acc
        // layout is the A operand of -N_i L; then T = (-N_i L) N_{i-1}.  fp32 products as
        // hi / lo passes; T goes to LDS transposed, like N.
        auto t_blocks = [&](int b) {
            if constexpr (FAM == FAM_GDN && NTC == 4) {
                const bf16* LT = sLT(b);
                const bf16* NT = sNT(b);
                bf16* TT = sTT(b);
                constexpr int JL[2] = {off_index(1, 0), off_index(3, 2)};
                f32x4 y[2];
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    const int i = 2 * q + 1, j = JL[q];
                    // (-L)^T as A: (-L)[4g+r][c] = XT[c][4g+r], a plain read of XT row c
                    const bf16x4 lh = lds4(LT + j * BLK + c16 * SB + 4 * g);
                    const bf16x4 ll = lds4(LT + (NOFF + j) * BLK + c16 * SB + 4 * g);
                    // N_i^T as B: N_i[c][4g+r] = NT[4g+r][c], a transposed read
                    const bf16x4 nh = lds4_tr(NT + i * BLK, SB, 0, 0, g, c16);
                    const bf16x4 nl = lds4_tr(NT + (NTC + i) * BLK, SB, 0, 0, g, c16);
                    f32x4 acc = mma16(lh, nh, zero4());
                    acc = mma16(lh, nl, acc);
                    y[q] = mma16(ll, nh, acc);
                }
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    const int i = 2 * q + 1;
                    // N_{i-1} as B: N[4g+r][c] = NT[c][4g+r], a plain read
                    const bf16x4 nh = lds4(NT + (i - 1) * BLK + c16 * SB + 4 * g);
                    const bf16x4 nl = lds4(NT + (NTC + i - 1) * BLK + c16 * SB + 4 * g);
                    const Split4 ys = split4(y[q]);
                    f32x4 t = mma16(ys.hi, nh, zero4());
                    t = mma16(ys.hi, nl, t);
                    t = mma16(ys.lo, nh, t);
                    store_tile_tr<SB, true>(TT + q * BLK, 2 * BLK, t, g, c16);
                }
            }
        };

        // A-waves, second phase: state-independent blocks of chunk ci into buffer ci & 1
        auto a_work = [&](int ci) {
            const int b = ci & 1;
            if (FAM == FAM_GDN && !stager) {
                // the solver: wait until every stager has masked its diagonal blocks
                // of chunk ci (NSTG signals per chunk), then invert them
                const bool ok = lds_wait_count(diag_cnt, (uint32_t)(NSTG * (ci + 1)), p.wait_limit);
                diag_solve_all(b, ok);
                return;
            }
            // this wave's gate prefix row (gate_rows, one barrier earlier)
            const float* gcw = reinterpret_cast<const float*>(smem + Ly::GC_OFF) + 64 * wa;
            using NS = integral_constant<int, NSTG>;
            if constexpr (FAM == FAM_GDN) {
                // stager a masks its diagonal blocks and signals the solver, then
                // builds the strictly-lower L blocks a, a + NSTG, ...
                static_assert(NSTG == 3, "three stagers");
                switch (wa) {
                    case 0:
                        diag_prep(integral_constant<int, 2>(), b, gcw);
                        lds_signal(diag_cnt, lane);
                        items(integral_constant<int, 0>(), NS(), L_KIND(), b, gcw);
                        break;
                    case 1:
                        diag_prep(integral_constant<int, 1>(), b, gcw);
                        lds_signal(diag_cnt, lane);
                        items(integral_constant<int, 1>(), NS(), L_KIND(), b, gcw);
                        break;
                    default:
                        diag_prep(integral_constant<int, 0>(), b, gcw);
                        lds_signal(diag_cnt, lane);
                        items(integral_constant<int, 2>(), NS(), L_KIND(), b, gcw);
                        break;
                }
            } else if (with_out) {
                // Mamba-2: stager a builds the output blocks P a, a + NSTG, ... (these
                // waves are otherwise idle in this phase)
                static_assert(NSTG == 4, "four stagers");
                switch (wa) {
                    case 0: items(integral_constant<int, 0>(), NS(), P_KIND(), b, gcw); break;
                    case 1: items(integral_constant<int, 1>(), NS(), P_KIND(), b, gcw); break;
                    case 2: items(integral_constant<int, 2>(), NS(), P_KIND(), b, gcw); break;
                    default: items(integral_constant<int, 3>(), NS(), P_KIND(), b, gcw); break;
                }
            }
        };

        // prologue: chunk 0 staged and its blocks built; chunk 1 in flight.  While
        // the B-waves run chunk c, the stagers commit chunk c+1 (loaded during
        // chunk c-1), issue the loads of chunk c+2, and mask chunk c+1's diagonal
        // blocks and build its L blocks (Mamba-2: its P blocks), Gated DeltaNet
        // committing q and v of chunk c+1 after those blocks; the solver forms
        // chunk c's T blocks, then inverts chunk c+1's diagonal blocks.
        // The stagers and the solver also run separate loops (same barrier
        // sequence), so the solver's registers do not overlap the prefetch ones.
        if (stager) {
            if (nch > 0) {
                prefetch(0);
                if (QV_LATE) prefetch_qv(0);
                commit(0);
                if (QV_LATE) commit_qv(0);
                gate_rows(0);
            }
            chunk_barrier();
            if (nch > 0) {
                a_work(0);
                if (nch > 1) {
                    prefetch(1);
                    if (QV_LATE) prefetch_qv(1);
                }
            }
            for (int ci = 0; ci < nch; ++ci) {
                chunk_barrier();
                if (ci + 1 < nch) {
                    commit(ci + 1);
                    gate_rows(ci + 1);
                }
                if (ci + 2 < nch) prefetch(ci + 2);  // a whole chunk of lead time
                chunk_barrier();
                if (ci + 1 < nch) {
                    a_work(ci + 1);
                    // q / v of chunk ci+1: first read after the next barrier; their
                    // buffer was last read in chunk ci-1
                    if (QV_LATE) commit_qv(ci + 1);
                }
                if (QV_LATE && ci + 2 < nch) prefetch_qv(ci + 2);
            }
        } else {
            chunk_barrier();
            if (nch > 0) a_work(0);
            for (int ci = 0; ci < nch; ++ci) {
                chunk_barrier();
                // chunk ci's T blocks (its diagonal inverses and L blocks were built
                // before the barrier), needed by the B-waves after the next barrier
                t_blocks(ci & 1);
                chunk_barrier();
                if (ci + 1 < nch) a_work(ci + 1);
            }
        }
        if (FAM == FAM_SSD && SUMMARY && p.M_out && tile == 0 && wa == 0 && lane == 0)
            p.M_out[int64_t(s) * p.h_v + h] = lam_sum;
    }
}

hipError_t launch_scan_gdn(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st);
hipError_t launch_scan_ssd(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st);
size_t scan_lds_bytes(int fam, int dk, int chunk, bool f32io, int nb, bool summary);
// Mamba-2 scan / block-summary kernel with eight symmetric state waves, and
// the output correction of its pieces (ssd_scan.hip)
bool ssd_scan_supported(int dk, int chunk, bool f32io, int dv);
hipError_t launch_ssd_scan(int dk, const ScanArgs& a, hipStream_t st);
struct SsdCorrectArgs {
    const int32_t* cu;     // the requests' token ranges (as the scan's cu)
    int32_t n_seq;
    int64_t n_tok;
    const void* C;         // [n_tok, h_qk, dk] bf16
    const float* dt;       // [n_tok, h_v]
    const float* A;        // [h_v]
    int32_t h_qk, h_v, dv, pieces;
    const float* piece_B;  // the pieces' end states and log-decay sums (ScanArgs::piece_B / piece_L)
    const float* piece_L;
    void* y;               // [n_tok, h_v, dv] bf16: piece outputs from zero, corrected in place; or null
    float* S_final;        // [n_seq, h_v, dv, dk] or null
    int32_t tiles;         // 64-row tiles over dv
    int32_t slots;         // chunk slots per piece (1..8): slot j takes chunks j, j + slots, ...
    int32_t n_units;
};
hipError_t launch_ssd_correct(int dk, const SsdCorrectArgs& a, hipStream_t st);

template <int FAM, int DK, int CH, bool F32IO, int NB, bool SUMMARY, int RT = 1>
hipError_t launch_chunk_nb(const ScanArgs& a, hipStream_t st) {
    const size_t lds = ChunkLds<FAM, DK, CH, F32IO, NB * RT, SUMMARY>::BYTES;
    auto kern = chunk_kernel<FAM, DK, CH, F32IO, NB, SUMMARY, RT>;
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
        case 8:
            // a whole 128-row transition per workgroup: the state-independent work of
            // a chunk is shared by four state waves of two row tiles each, which
            // also share every K fragment they read
            if constexpr (SUMMARY && DK == 128 && CH == 64 && !F32IO)
                return launch_chunk_nb<FAM, DK, CH, F32IO, 4, SUMMARY, 2>(a, st);
            return hipErrorInvalidValue;
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
        case 17: return (DK == 128 && CH == 64 && !F32IO) ? ChunkLds<FAM, DK, CH, F32IO, 8, true>::BYTES : 0;
    }
    return 0;
}

}  // namespace lkv
