// Mamba-2 (SSD) online scan and block summary.  Per chunk of CH tokens, with
// the in-chunk cumulative log-decay l_t = A_h * sum dt (Eq. 2's scalar decay),
// d_t = dt_t exp(l_C - l_t) and the output blocks
// P = lower(exp(l_t - l_i) * C B^T) diag(dt):
//   y^T = diag(exp(l)) (S C^T) + X^T P^T        (outputs, transposed tiles)
//   S   <- exp(l_C) S + X^T diag(d) B            (Eq. 5 over the chunk)
// The state enters no product but the output's S C^T, whose result only feeds
// the bf16 output, so the state is split into its bf16 hi part alone; the
// update's fp32 operand d * X is split hi / lo (two passes onto the fp32 state).
//
// Nothing of a chunk waits on a triangular solve, so the waves of a workgroup
// work alike.  A wave issues about one LDS read per 30 cycles whatever its
// width (measured on gfx950), and the CU's LDS serves 128 B per cycle: four
// waves saturate it with 16-byte reads, eight with the 8-byte transposed reads
// most of the fragments here need.  So the 64 state rows of a work unit are
// spread over eight waves: wave w owns row tile w % 4 and half
// w / 4 of the dk columns of the state (its update), and forms the outputs of
// token half w / 4 of its row tile from the whole row tile's hi parts, half of
// which its partner wave hands over through LDS after every update.
//
// Work unit = (segment, head, tile of 64 state rows).  Per chunk: two LDS-only
// workgroup barriers; chunk c+1's tiles are committed and its output blocks
// built while chunk c is used (two LDS buffers), chunk c+2's tiles are loaded
// into registers a whole chunk ahead through buffer resources that end at the
// segment's end (rows past it read as zero).  The products are issued in the
// order of the shared chunk kernel's Mamba-2 path, so both give identical bits.
#include "chunk_kernel.h"

namespace lkv {

// Piece pc of P of the token range [t0, t1): pieces of whole chunks, ceil(len /
// P) tokens rounded up to a chunk multiple each; the last pieces take what is
// left and may be empty (the sequence-parallel scan's cut).
__device__ __forceinline__ void piece_range(int64_t& t0, int64_t& t1, int P, int pc, int CH) {
    const int64_t len = t1 - t0;
    const int64_t per = ((len + P - 1) / P + CH - 1) / CH * CH;
    const int64_t a = (int64_t)pc * per, b = a + per;
    t1 = t0 + (b < len ? b : len);
    t0 = t0 + (a < len ? a : len);
}

template <int DK>
struct SsdLds {
    static constexpr int CH = 64, NTC = 4, NTK = DK / 16, NH = NTK / 2;
    static constexpr int SK = DK + 16;  // kq_pos rows of B and C (conflict-free fragment reads)
    static constexpr int SX = 64 + 8;   // X rows: this tile's 64 state rows
    static constexpr int SB = 20, BLK = 16 * SB;
    static constexpr int NPB = NTC * (NTC + 1) / 2;  // lower 16x16 output blocks
    static __host__ __device__ constexpr size_t al(size_t x) { return (x + 15) & ~size_t(15); }
    static constexpr size_t B_OFF = 0;
    static constexpr size_t C_OFF = B_OFF + al(size_t(CH) * SK * 2);
    static constexpr size_t X_OFF = C_OFF + al(size_t(CH) * SK * 2);
    // gate rows: dt | l | exp(l) | d | exp(l_C), l_C
    static constexpr size_t G_OFF = X_OFF + al(size_t(CH) * SX * 2);
    static constexpr size_t P_OFF = G_OFF + al((4 * CH + 4) * 4);
    static constexpr size_t BUF = P_OFF + al(size_t(NPB) * BLK * 2);
    // state hi parts handed between the two waves of a row tile: [2][4 row
    // tiles][NTK dk tiles][64 lanes] x 4 bf16, each lane's own acc-tile values
    static constexpr size_t SH_OFF = 2 * BUF;
    static constexpr size_t SH_BUF = size_t(4) * NTK * 64 * 8;
    static constexpr size_t BYTES = SH_OFF + 2 * SH_BUF;
};

template <int DK>
__global__ __launch_bounds__(512) void ssd_scan_kernel(ScanArgs p) {
    using Ly = SsdLds<DK>;
    constexpr int CH = Ly::CH, NTC = Ly::NTC, NTK = Ly::NTK, NH = Ly::NH;
    constexpr int SK = Ly::SK, SX = Ly::SX, SB = Ly::SB, BLK = Ly::BLK, NPB = Ly::NPB;
    extern __shared__ __align__(16) char smem[];
    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63, g = lane >> 4, c16 = lane & 15;
    const int rt = w & 3;   // row tile of this wave
    const int hf = w >> 2;  // its dk half (state, update) and token half (outputs)

    // ---- work unit: row tiles innermost, then heads (adjacent heads of one
    // group read the same B and C rows: one XCD's L2), then the segment
    const int tiles = p.tiles_b;
    const int u = xcd_unit(blockIdx.x, p.n_units);
    const int tile = u % tiles;
    const int h = (u / tiles) % p.h_v;
    const int sp = u / (tiles * p.h_v);  // segment, or (segment, piece) with pieces > 1
    const int P = p.pieces > 1 ? p.pieces : 1;
    const int s = sp / P, pc = sp % P;
    const int hq = h / (p.h_v / p.h_qk);
    const int row0 = tile * 64;
    const int my_row = row0 + 16 * rt + c16;  // the state row this lane's tiles hold
    int64_t t0 = p.cu[s], t1 = p.cu[s + 1];
    t0 = t0 < 0 ? 0 : (t0 > p.n_tok ? p.n_tok : t0);
    t1 = t1 < t0 ? t0 : (t1 > p.n_tok ? p.n_tok : t1);
    if (P > 1) piece_range(t0, t1, P, pc, CH);
    const int nch = (int)((t1 - t0 + CH - 1) / CH);
    const float Ah = p.A[h];

    auto sB = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::B_OFF); };
    auto sC = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::C_OFF); };
    auto sX = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::X_OFF); };
    auto sG = [&](int b) { return reinterpret_cast<float*>(smem + b * Ly::BUF + Ly::G_OFF); };
    auto sP = [&](int b) { return reinterpret_cast<bf16*>(smem + b * Ly::BUF + Ly::P_OFF); };
    // hi-part exchange slot of dk tile nt of this row tile, buffer e
    auto sSh = [&](int e, int nt) {
        return reinterpret_cast<bf16x4*>(smem + Ly::SH_OFF + e * Ly::SH_BUF) + (rt * NTK + nt) * 64 + lane;
    };

    // ---- chunk tiles: registers (a chunk ahead) -> LDS
    KQTile<CH, DK, false, 512> pB, pC;
    TileRegs<CH, 64, false, 512> pX;
    uint32_t pdt = 0u;  // wave 0: lane t's dt, raw bits until its commit
    float lam = 0.f;    // wave 0: the segment's log-decay sum so far (block summaries' Lambda)
    const bool with_out = p.out != nullptr;
    const uint32_t bc_rb = (uint32_t)p.h_qk * DK * 2, x_rb = (uint32_t)p.h_v * p.dv * 2;
    auto prefetch = [&](int ci) {
        const int64_t c0 = t0 + (int64_t)ci * CH;
        const uint32_t n = (uint32_t)((t1 - c0) < CH ? (t1 - c0) : CH);
        const int64_t bc_off = (c0 * p.h_qk + hq) * (int64_t)DK * 2;
        pB.load_buf(make_rsrc(reinterpret_cast<const char*>(p.k) + bc_off, n * bc_rb), 0u, bc_rb, tid);
        if (with_out) pC.load_buf(make_rsrc(reinterpret_cast<const char*>(p.q) + bc_off, n * bc_rb), 0u, bc_rb, tid);
        pX.load_buf(make_rsrc(reinterpret_cast<const char*>(p.v) + ((c0 * p.h_v + h) * (int64_t)p.dv + row0) * 2,
                              n * x_rb),
                    0u, x_rb, tid);
        if (w == 0) {
            const uint32_t g_rb = (uint32_t)p.h_v * 4;
            pdt = buf_load4(make_rsrc(reinterpret_cast<const char*>(p.g) + (c0 * p.h_v + h) * 4, n * g_rb),
                            (uint32_t)lane * g_rb);
        }
    };
    // commit, and (wave 0) the chunk's gate rows from its dt registers
    auto commit = [&](int ci) {
        const int b = ci & 1;
        pB.commit(sB(b), SK, 0, tid);
        if (with_out) pC.commit(sC(b), SK, 0, tid);
        pX.commit(sX(b), SX, 0, tid);
        if (w == 0) {
            float* G = sG(b);
            const float dt = __builtin_bit_cast(float, pdt);
            const float l = wave_incl_scan(Ah * dt);  // lanes past the segment hold dt = 0
            const float lC = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, l), CH - 1));
            G[lane] = dt;
            G[CH + lane] = l;
            G[2 * CH + lane] = __expf(l);
            G[3 * CH + lane] = dt * __expf(lC - l);
            lam += lC;
            if (lane == 0) {
                G[4 * CH] = __expf(lC);
                G[4 * CH + 1] = lC;
            }
        }
    };
    // the output blocks P[t][i] = exp(l_t - l_i) (C_t . B_i) dt_i, i <= t, of one
    // chunk, stored transposed (bf16) for direct fragment reads.  Wave w builds
    // blocks (mt, nt0) and (mt, nt0 + 1) of one row block, so that they share
    // the C fragments: (3,0-1) (3,2-3) (2,0-1) (2,2) (1,0-1) (0,0); waves 6 and
    // 7 build none.  LDS reads are what bounds a chunk, and this order reads 64
    // fragment rows where one block per wave would read 80.
    auto p_blocks = [&](int b) {
        const int mt = w < 2 ? 3 : w < 4 ? 2 : w == 4 ? 1 : 0;
        const int nt0 = w < 4 ? 2 * (w & 1) : 0;
        const int nb = w >= 6 ? 0 : (w == 3 || w == 5) ? 1 : 2;
        if (nb == 0) return;
        const bf16* Cb = sC(b) + (16 * mt + c16) * SK + 8 * g;
        const bf16* Bb = sB(b) + (16 * nt0 + c16) * SK + 8 * g;
        const float* G = sG(b);
        // every fragment is requested before the first product: a chunk is bound
        // by LDS latency wherever products wait on reads one slice at a time
        constexpr int NKP = NTK / 2;
        bf16x8 fa[NKP], fb0[NKP], fb1[NKP];
#pragma unroll
        for (int kp = 0; kp < NKP; ++kp) {
            fa[kp] = lds8(Cb + 32 * kp);
            fb0[kp] = lds8(Bb + 32 * kp);
            fb1[kp] = lds8(Bb + 16 * SK + 32 * kp);  // in the tile for every wave; unused when nb = 1
        }
        __builtin_amdgcn_sched_barrier(0);
        f32x4 acc[2] = {zero4(), zero4()};
#pragma unroll
        for (int kp = 0; kp < NKP; ++kp) {
            acc[0] = mma32(fa[kp], fb0[kp], acc[0]);
            acc[1] = mma32(fa[kp], fb1[kp], acc[1]);
        }
        const f32x4 lt = lds4f(G + CH + 16 * mt + 4 * g);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            if (i >= nb) break;  // wave-uniform
            const int nt = nt0 + i;
            const int ic = 16 * nt + c16;
            const float li = G[CH + ic], dti = G[ic];
            f32x4 v;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float e = dti * __expf(lt[r] - li) * acc[i][r];
                v[r] = (mt > nt || c16 <= 4 * g + r) ? e : 0.f;
            }
            store_tile_tr<SB, false>(sP(b) + low_index(mt, nt) * BLK, NPB * BLK, v, g, c16);
        }
    };

    // chunk 0's tiles are requested first; the initial state's loads follow
    if (nch > 0) prefetch(0);

    // ---- this wave's half of the state: S[j] holds S[my_row][16 (NH hf + j) + 4g + r]
    f32x4 S[NH];
    {
        int64_t init_row = s;
        float init_fill = 0.f;
        bool init_load = p.S_init != nullptr && pc == 0;  // later pieces start from zero
        if (p.src && pc == 0) {
            const int32_t id = p.src[s];
            init_row = id;
            if (id < 0 || id >= p.n_src) {
                init_load = false;
                init_fill = id == -1 ? 0.f : __builtin_nanf("");
            }
        }
        // one branch for the whole half tile, so that all its loads are in flight together
        const int64_t e0 = ((init_row * p.h_v + h) * p.dv + my_row) * DK + 16 * NH * hf + 4 * g;
        if (init_load && p.init_bf16) {
            uint2 q[NH];
#pragma unroll
            for (int j = 0; j < NH; ++j)
                q[j] = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(p.S_init) + e0 + 16 * j);
#pragma unroll
            for (int j = 0; j < NH; ++j) S[j] = to_f32(__builtin_bit_cast(bf16x4, q[j]));
        } else if (init_load) {
#pragma unroll
            for (int j = 0; j < NH; ++j) S[j] = *reinterpret_cast<const f32x4*>(p.S_init + e0 + 16 * j);
        } else {
#pragma unroll
            for (int j = 0; j < NH; ++j) S[j] = f32x4{init_fill, init_fill, init_fill, init_fill};
        }
    }
    const bf16x8 negI = neg_eye(g, c16);
    // hi parts of this half, kept for the next outputs and handed to the partner
    bf16x4 Sh[NH];
    auto publish = [&](int e) {
#pragma unroll
        for (int j = 0; j < NH; ++j) {
            Sh[j] = to_bf16(S[j]);
            *sSh(e, NH * hf + j) = Sh[j];
        }
    };
    // The initial state is used here on every path, so its loads are complete
    // before the loop: a state register still waiting on a load at the loop
    // head would make the loop's first use of the state wait for every load in
    // flight -- the next chunk's prefetch included -- in every chunk.
#pragma unroll
    for (int j = 0; j < NH; ++j) Sh[j] = to_bf16(S[j]);
    if (with_out) {
#pragma unroll
        for (int j = 0; j < NH; ++j) *sSh(0, NH * hf + j) = Sh[j];
    }

    // ---- prologue: chunk 0 committed, its output blocks built; chunk 1 in flight
    if (nch > 0) {
        commit(0);
        if (nch > 1) prefetch(1);
    }
    lds_barrier();
    if (nch > 0 && with_out) p_blocks(0);

    // outputs of token half HF of this row tile: y^T tile mt = exp(l_t) S C^T + X^T P^T
    auto outputs = [&](auto hf_c, int b, int e, int64_t c0, int n, const bf16x4* Xf) {
        constexpr int HF = decltype(hf_c)::value;
        constexpr int NKP = NTK / 2;
        constexpr int J0 = HF == 0 ? 0 : 3, NJ = HF == 0 ? 3 : 7;  // output blocks of token tiles 2HF, 2HF+1
        const float* G = sG(b);
        const bf16* Cb = sC(b);
        // every operand is requested before the first product: the row tile's hi
        // parts (this wave's half from registers, the partner's from LDS), the C
        // fragments, the output blocks and the decay factors
        bf16x4 Sf[NTK];
#pragma unroll
        for (int nt = 0; nt < NTK; ++nt) Sf[nt] = (nt / NH == HF) ? Sh[nt % NH] : *sSh(e, nt);
        bf16x8 cf[NKP][2];
#pragma unroll
        for (int kp = 0; kp < NKP; ++kp)
#pragma unroll
            for (int m = 0; m < 2; ++m) cf[kp][m] = lds8(Cb + (16 * (2 * HF + m) + c16) * SK + 32 * kp + 8 * g);
        bf16x4 Pf[NJ];
#pragma unroll
        for (int j = 0; j < NJ; ++j) Pf[j] = lds4_tr(sP(b) + (J0 + j) * BLK, SB, 0, 0, g, c16);
        float el[2];
#pragma unroll
        for (int m = 0; m < 2; ++m) el[m] = G[2 * CH + 16 * (2 * HF + m) + c16];
        __builtin_amdgcn_sched_barrier(0);
        f32x4 OT[2];
#pragma unroll
        for (int m = 0; m < 2; ++m) OT[m] = zero4();
#pragma unroll
        for (int kp = 0; kp < NKP; ++kp)
#pragma unroll
            for (int m = 0; m < 2; ++m) OT[m] = mma32(Sf[2 * kp], Sf[2 * kp + 1], cf[kp][m], OT[m]);
#pragma unroll
        for (int m = 0; m < 2; ++m) OT[m] *= el[m];
        // tile mt contracts over token blocks 0..mt, pairs of blocks per product
#pragma unroll
        for (int kp = 0; kp < NTC; kp += 2) {
#pragma unroll
            for (int m = 0; m < 2; ++m) {
                const int mt = 2 * HF + m;
                if (mt < kp) continue;
                const bool two = mt >= kp + 1;
                const int j0 = low_index(mt, kp) - J0;
                const bf16x4 p1 = two ? Pf[j0 + 1] : zero_bf16x4();
                const bf16x4 x1 = two ? Xf[kp + 1] : zero_bf16x4();
                OT[m] = mma32(Xf[kp], x1, Pf[j0], p1, OT[m]);
            }
        }
        const int64_t rowcol = (int64_t)h * p.dv + row0 + 16 * rt + 4 * g;
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            const int t = 16 * (2 * HF + m) + c16;
            if (t < n) {
                const int64_t oi = (c0 + t) * p.h_v * (int64_t)p.dv + rowcol;
                *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(p.out) + oi) = to_bf16(OT[m]);
            }
        }
    };

    for (int ci = 0; ci < nch; ++ci) {
        const int b = ci & 1;
        const int64_t c0 = t0 + (int64_t)ci * CH;
        const int n = (int)((t1 - c0) < CH ? (t1 - c0) : CH);
        lds_barrier();  // chunk ci's blocks built and the partner's hi parts published; buffer b ^ 1 free
        if (ci + 1 < nch) commit(ci + 1);
        if (ci + 2 < nch) prefetch(ci + 2);  // a whole chunk of lead time
        const float* G = sG(b);
        // X fragments of this row tile (A operand of X^T P^T, the B side of the
        // update): lane (g, c) holds X[16kt + 4g + j][16 rt + c]
        bf16x4 Xf[NTC];
#pragma unroll
        for (int kt = 0; kt < NTC; ++kt) Xf[kt] = lds4_tr(sX(b), SX, 16 * kt, 16 * rt, g, c16);
        if (with_out) {
            if (hf == 0) outputs(std::integral_constant<int, 0>(), b, ci & 1, c0, n, Xf);
            else outputs(std::integral_constant<int, 1>(), b, ci & 1, c0, n, Xf);
        }
        // S <- exp(l_C) S + B^T diag(d) X on this wave's dk half: the fp32
        // operand d * X as hi / lo passes
        bf16x4 Wh[NTC], Wl[NTC];
#pragma unroll
        for (int kt = 0; kt < NTC; ++kt) {
            const f32x4 d = lds4f(G + 3 * CH + 16 * kt + 4 * g);
            const Split4 sp = split4_mm(d * to_f32(Xf[kt]), negI);
            Wh[kt] = sp.hi;
            Wl[kt] = sp.lo;
        }
        const float aC = G[4 * CH];
#pragma unroll
        for (int j = 0; j < NH; ++j) S[j] = aC * S[j];
        const bf16* Bb = sB(b);
        bf16x4 x0[2][NH], x1[2][NH];
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
            for (int j = 0; j < NH; ++j) {
                x0[q][j] = lds4_tr_kq<DK>(Bb, SK, 32 * q, 16 * (NH * hf + j), g, c16);
                x1[q][j] = lds4_tr_kq<DK>(Bb, SK, 32 * q + 16, 16 * (NH * hf + j), g, c16);
            }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
            for (int j = 0; j < NH; ++j) {
                S[j] = mma32(x0[q][j], x1[q][j], Wh[2 * q], Wh[2 * q + 1], S[j]);
                S[j] = mma32(x0[q][j], x1[q][j], Wl[2 * q], Wl[2 * q + 1], S[j]);
            }
        if (with_out) publish((ci + 1) & 1);
        lds_barrier();  // chunk ci+1 committed
        if (ci + 1 < nch && with_out) p_blocks(b ^ 1);
    }
    if (p.summary && p.M_out && tile == 0 && w == 0 && lane == 0) p.M_out[int64_t(s) * p.h_v + h] = lam;
    float* dst = P > 1 ? p.piece_B : p.S_final;
    if (P > 1 && tile == 0 && w == 0 && lane == 0) p.piece_L[int64_t(sp) * p.h_v + h] = lam;
    if (dst) {
#pragma unroll
        for (int j = 0; j < NH; ++j)
            *reinterpret_cast<f32x4*>(dst + ((int64_t(sp) * p.h_v + h) * p.dv + my_row) * DK + 16 * (NH * hf + j) +
                                      4 * g) = S[j];
    }
}

// Output correction of the sequence-parallel Mamba-2 scan.  With a scalar
// decay per token the state at token t of piece p is exp(L_t) S_p + (the state
// of the piece's own tokens from zero), L_t being the log-decay summed from
// the piece's start through t (Eq. 2).  So the outputs of a piece scanned from
// zero lack exactly exp(L_t) C_t S_p^T, and its start state S_p is Eq. 5 over
// the earlier pieces: S_1 = (piece 0's end state, which started from the
// request's own), S_{p+1} = exp(Lambda_p) S_p + B_p.  One workgroup per
// (request, piece >= 1, head, 64 state rows, chunk slot j of J), four waves of
// 16 rows: it composes S_p (slot 0 of the last piece also the final state),
// then takes the piece's chunks j, j + J, ... adding exp(L_t) (S_p C^T) to
// their outputs.  The slots put a piece's chunks in flight together: each
// chunk is little work, and a workgroup waiting on one load round trip per
// chunk would be bound by memory latency.  S_p enters the product as its bf16
// hi part, like the state in the scan's own outputs.
template <int DK>
__global__ __launch_bounds__(256) void ssd_correct_kernel(SsdCorrectArgs p) {
    constexpr int CH = 64, NTC = 4, NTK = DK / 16, SK = DK + 16, JMAX = 8;
    extern __shared__ __align__(16) char smem[];
    bf16* sC = reinterpret_cast<bf16*>(smem);
    float* sE = reinterpret_cast<float*>(smem + size_t(CH) * SK * 2);  // exp(L_t) of the chunk's tokens
    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63, g = lane >> 4, c16 = lane & 15;
    const int P = p.pieces, J = p.slots;
    // unit order, innermost first: chunk slot, row tile, head, (request, piece)
    const int u = xcd_unit(blockIdx.x, p.n_units);
    const int j = u % J;
    const int tile = (u / J) % p.tiles;
    const int h = (u / (J * p.tiles)) % p.h_v;
    const int rp = u / (J * p.tiles * p.h_v);
    const int r = rp / (P - 1), pc = rp % (P - 1) + 1;
    const int hq = h / (p.h_v / p.h_qk);
    const int row0 = tile * 64;
    const int my_row = row0 + 16 * w + c16;
    int64_t t0 = p.cu[r], t1 = p.cu[r + 1];
    t0 = t0 < 0 ? 0 : (t0 > p.n_tok ? p.n_tok : t0);
    t1 = t1 < t0 ? t0 : (t1 > p.n_tok ? p.n_tok : t1);
    piece_range(t0, t1, P, pc, CH);
    const int nch = (int)((t1 - t0 + CH - 1) / CH);
    const bool outputs = p.y != nullptr && j < nch;  // uniform over the workgroup
    const bool final_state = pc == P - 1 && j == 0 && p.S_final != nullptr;
    if (!outputs && !final_state) return;

    // ---- this slot's first chunk is requested before the start state: the C
    // tile and dt a chunk ahead in registers, the outputs being corrected too
    KQTile<CH, DK, false, 256> pCt;
    uint32_t pdt = 0u;  // wave 0: the chunk's dt (lane = token)
    float pskip = 0.f;  // wave 0: dt summed over the chunks this slot skips next
    bf16x4 py[NTC];
    const float Ah = p.A[h];
    const uint32_t c_rb = (uint32_t)p.h_qk * DK * 2, g_rb = (uint32_t)p.h_v * 4;
    const int64_t ycol_w = (int64_t)h * p.dv + row0 + 16 * w;  // the wave's first output row (uniform)
    const int64_t ycol = ycol_w + 4 * g;
    // dt of the piece's tokens from t0: zero past the piece
    const __amdgpu_buffer_rsrc_t rdt =
        make_rsrc(reinterpret_cast<const char*>(p.dt) + (t0 * p.h_v + h) * 4, (uint32_t)(t1 - t0) * g_rb);
    auto prefetch = [&](int ci) {
        const int64_t c0 = t0 + (int64_t)ci * CH;
        const uint32_t n = (uint32_t)((t1 - c0) < CH ? (t1 - c0) : CH);
        pCt.load_buf(make_rsrc(reinterpret_cast<const char*>(p.C) + (c0 * p.h_qk + hq) * (int64_t)DK * 2, n * c_rb), 0u,
                     c_rb, tid);
        if (w == 0) {
            pdt = buf_load4(rdt, (uint32_t)(ci * CH + lane) * g_rb);
            float acc = 0.f;
#pragma unroll
            for (int k = 1; k < JMAX; ++k) {
                const uint32_t off = k < J ? (uint32_t)((ci + k) * CH + lane) * g_rb : 0xffffffffu;
                acc += __builtin_bit_cast(float, buf_load4(rdt, off));
            }
            pskip = acc;
        }
        // this lane's outputs: 4 rows of token 16mt + c16 (zeros past the piece);
        // the resource's base is the wave's (uniform), the lane's rows in the offset
        const uint32_t y_rb = (uint32_t)p.h_v * p.dv * 2;
        const __amdgpu_buffer_rsrc_t ry =
            make_rsrc(reinterpret_cast<const char*>(p.y) + (c0 * p.h_v * (int64_t)p.dv + ycol_w) * 2, n * y_rb);
#pragma unroll
        for (int mt = 0; mt < NTC; ++mt) {
            const uint32_t t = 16 * mt + c16;
            const uint32_t off = t < n ? t * y_rb + 8 * g : 0xffffffffu;
            py[mt] = __builtin_bit_cast(bf16x4, __builtin_amdgcn_raw_buffer_load_b64(ry, off, 0, 0));
        }
    };
    float Lrun = 0.f;  // wave 0: A_h times the piece's dt before the current chunk
    if (outputs) {
        prefetch(j);
        if (w == 0) {
            // the chunks before this slot's first one (j < JMAX), all requested at once
            float acc = 0.f;
#pragma unroll
            for (int k = 0; k < JMAX - 1; ++k) {
                const uint32_t off = k < j ? (uint32_t)(k * CH + lane) * g_rb : 0xffffffffu;
                acc += __builtin_bit_cast(float, buf_load4(rdt, off));
            }
            Lrun = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, wave_incl_scan(Ah * acc)),
                                                                          CH - 1));
        }
    }

    // ---- the piece's start state (acc layout: S[nt] holds S[my_row][16nt + 4g + r])
    // as the weighted sum S_p = sum_q exp(Lambda_{q+1} + ... + Lambda_{p-1}) B_q,
    // four pieces' states requested at a time (one load round trip for p <= 4)
    auto brow = [&](int q) {
        return p.piece_B + ((int64_t(r) * P + q) * p.h_v + h) * (int64_t)p.dv * DK + (int64_t)my_row * DK + 4 * g;
    };
    auto lam = [&](int q) { return p.piece_L[(int64_t(r) * P + q) * p.h_v + h]; };
    // lane q: the log-weight of piece q's state (pieces past pc: unused)
    float lw;
    {
        const float x = (lane >= 1 && lane < pc) ? lam(lane) : 0.f;
        const float pre = wave_incl_scan(x);
        const float tot = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, pre), CH - 1));
        lw = tot - pre;
    }
    f32x4 S[NTK];
#pragma unroll
    for (int nt = 0; nt < NTK; ++nt) S[nt] = zero4();
    for (int q0 = 0; q0 < pc; q0 += 4) {  // pc <= P - 1 < 64
        f32x4 bl[4][NTK];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if (q0 + i >= pc) break;  // uniform
            const float* bq = brow(q0 + i);
#pragma unroll
            for (int nt = 0; nt < NTK; ++nt) bl[i][nt] = *reinterpret_cast<const f32x4*>(bq + 16 * nt);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if (q0 + i >= pc) break;  // uniform
            const float e = __expf(__builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, lw),
                                                                                         q0 + i)));
#pragma unroll
            for (int nt = 0; nt < NTK; ++nt) S[nt] += e * bl[i][nt];
        }
    }
    if (final_state) {
        const float e = __expf(lam(pc));
        const float* bq = brow(pc);
        float* sf = p.S_final + ((int64_t(r) * p.h_v + h) * p.dv + my_row) * DK + 4 * g;
        f32x4 bl[NTK];  // every load in flight before the first store
#pragma unroll
        for (int nt = 0; nt < NTK; ++nt) bl[nt] = *reinterpret_cast<const f32x4*>(bq + 16 * nt);
#pragma unroll
        for (int nt = 0; nt < NTK; ++nt) *reinterpret_cast<f32x4*>(sf + 16 * nt) = e * S[nt] + bl[nt];
    }
    if (!outputs) return;
    bf16x4 Sh[NTK];
#pragma unroll
    for (int nt = 0; nt < NTK; ++nt) Sh[nt] = to_bf16(S[nt]);

    for (int ci = j; ci < nch; ci += J) {
        const int64_t c0 = t0 + (int64_t)ci * CH;
        const int n = (int)((t1 - c0) < CH ? (t1 - c0) : CH);
        lds_barrier();  // the previous chunk's tile is no longer read
        pCt.commit(sC, SK, 0, tid);
        if (w == 0) {
            const float l = wave_incl_scan(Ah * __builtin_bit_cast(float, pdt));  // zero dt past the piece
            sE[lane] = __expf(Lrun + l);
            const float skip = wave_incl_scan(Ah * pskip);
            Lrun += __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, l), CH - 1)) +
                    __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, skip), CH - 1));
        }
        bf16x4 yv[NTC];
#pragma unroll
        for (int mt = 0; mt < NTC; ++mt) yv[mt] = py[mt];
        if (ci + J < nch) prefetch(ci + J);
        lds_barrier();
        // y^T tile mt (rows 16w + 4g + j, tokens 16mt + c16) += exp(L_t) S_hi C^T
        constexpr int NKP = NTK / 2;
        bf16x8 cf[NKP][NTC];
#pragma unroll
        for (int kp = 0; kp < NKP; ++kp)
#pragma unroll
            for (int mt = 0; mt < NTC; ++mt) cf[kp][mt] = lds8(sC + (16 * mt + c16) * SK + 32 * kp + 8 * g);
        float el[NTC];
#pragma unroll
        for (int mt = 0; mt < NTC; ++mt) el[mt] = sE[16 * mt + c16];
        __builtin_amdgcn_sched_barrier(0);
        f32x4 OT[NTC];
#pragma unroll
        for (int mt = 0; mt < NTC; ++mt) OT[mt] = zero4();
#pragma unroll
        for (int kp = 0; kp < NKP; ++kp)
#pragma unroll
            for (int mt = 0; mt < NTC; ++mt) OT[mt] = mma32(Sh[2 * kp], Sh[2 * kp + 1], cf[kp][mt], OT[mt]);
#pragma unroll
        for (int mt = 0; mt < NTC; ++mt) {
            const int t = 16 * mt + c16;
            if (t < n) {
                const int64_t oi = (c0 + t) * p.h_v * (int64_t)p.dv + ycol;
                *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(p.y) + oi) =
                    to_bf16(to_f32(yv[mt]) + el[mt] * OT[mt]);
            }
        }
    }
}

template <int DK>
static hipError_t launch_ssd_correct_t(const SsdCorrectArgs& a, hipStream_t st) {
    const size_t lds = size_t(64) * (DK + 16) * 2 + 64 * 4;
    auto kern = ssd_correct_kernel<DK>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3(a.n_units), dim3(256), lds, st, a);
    return hipGetLastError();
}

hipError_t launch_ssd_correct(int dk, const SsdCorrectArgs& a, hipStream_t st) {
    switch (dk) {
        case 32: return launch_ssd_correct_t<32>(a, st);
        case 64: return launch_ssd_correct_t<64>(a, st);
        case 128: return launch_ssd_correct_t<128>(a, st);
    }
    return hipErrorInvalidValue;
}

template <int DK>
static hipError_t launch_ssd_scan_t(const ScanArgs& a, hipStream_t st) {
    const size_t lds = SsdLds<DK>::BYTES;
    auto kern = ssd_scan_kernel<DK>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3(a.n_units), dim3(512), lds, st, a);
    return hipGetLastError();
}

bool ssd_scan_supported(int dk, int chunk, bool f32io, int dv) {
    return !f32io && chunk == 64 && (dk == 32 || dk == 64 || dk == 128) && dv % 64 == 0;
}

hipError_t launch_ssd_scan(int dk, const ScanArgs& a, hipStream_t st) {
    switch (dk) {
        case 32: return launch_ssd_scan_t<32>(a, st);
        case 64: return launch_ssd_scan_t<64>(a, st);
        case 128: return launch_ssd_scan_t<128>(a, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace lkv
