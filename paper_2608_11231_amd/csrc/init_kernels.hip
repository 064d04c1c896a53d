// State initialisation kernels: single-block gather (Sec. 3.2) and exact
// composition of per-block (M, B) pairs (Eq. 5 applied block after block,
// which telescopes to Eq. 6).
#include "init_kernels.h"

#include <math.h>

namespace lkv {

// ---------------------------------------------------------------- pool rows
// Four consecutive pool elements widened to fp32: an fp32 pool is read as is, a
// bf16 pool (the cache's storage format) is widened exactly (bf16 -> fp32 only
// appends zero mantissa bits).
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <bool BF>
__device__ __forceinline__ f32x4 pool4(const void* base, int64_t elem) {
    if constexpr (BF) {
        const u32x2 u = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(
            reinterpret_cast<const uint16_t*>(base) + elem));
        return f32x4{__builtin_bit_cast(float, u.x << 16), __builtin_bit_cast(float, u.x & 0xffff0000u),
                     __builtin_bit_cast(float, u.y << 16), __builtin_bit_cast(float, u.y & 0xffff0000u)};
    } else {
        return __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(base) + elem));
    }
}

// ---------------------------------------------------------------- single block
// S_init[r] = B_pool[src[r]]: a bit-exact 16-byte-vector copy (or exact widening
// of a bf16 pool), HBM-bound.  One thread per four output elements; request
// r = index / per_req.
template <bool BF>
__global__ __launch_bounds__(256) void init_single_kernel(int32_t n_req, int32_t n_blk, int64_t per_req4,
                                                          const void* __restrict__ B_pool,
                                                          const int32_t* __restrict__ src,
                                                          f32x4* __restrict__ S) {
    const int64_t total = (int64_t)n_req * per_req4;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
        const int64_t r = i / per_req4, e = i - r * per_req4;
        const int32_t id = src[r];
        f32x4 v;
        if (id >= 0 && id < n_blk) {
            v = pool4<BF>(B_pool, 4 * ((int64_t)id * per_req4 + e));
        } else {
            const float f = (id == -1) ? 0.f : __builtin_nanf("");
            v = f32x4{f, f, f, f};
        }
        __builtin_nontemporal_store(v, S + i);
    }
}

hipError_t launch_init_single(int32_t n_req, int32_t n_blk, int64_t per_req, const void* B_pool, bool bf16_pool,
                              const int32_t* src, float* S, hipStream_t st) {
    const int64_t per4 = per_req / 4;
    const int64_t total = (int64_t)n_req * per4;
    if (total == 0) return hipSuccess;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 256 * 16) blocks = 256 * 16;
    if (bf16_pool)
        hipLaunchKernelGGL(init_single_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, st, n_req, n_blk,
                           per4, B_pool, src, reinterpret_cast<f32x4*>(S));
    else
        hipLaunchKernelGGL(init_single_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, st, n_req, n_blk,
                           per4, B_pool, src, reinterpret_cast<f32x4*>(S));
    return hipGetLastError();
}

// ---------------------------------------------------------------- Mamba-2 composition
// S <- B_{b_1}; S <- exp(Lambda_{b_j}) S + B_{b_j}.  Elementwise over the state.
// With S_steps, the state after each block but the request's last is also
// stored (request r's position j at row j - r).
template <bool BF>
__global__ __launch_bounds__(256) void compose_ssd_kernel(int32_t n_req, int32_t n_blk, int32_t H,
                                                          int64_t per_head4, const void* __restrict__ B_pool,
                                                          const float* __restrict__ Lam,
                                                          const int32_t* __restrict__ ids,
                                                          const int32_t* __restrict__ blk_cu, int32_t n_ids,
                                                          f32x4* __restrict__ S, f32x4* __restrict__ S_steps) {
    const int64_t total = (int64_t)n_req * H * per_head4;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
        const int64_t rh = i / per_head4, e = i - rh * per_head4;
        const int32_t r = (int32_t)(rh / H), h = (int32_t)(rh - (int64_t)r * H);
        int32_t b0 = blk_cu[r], b1 = blk_cu[r + 1];
        b0 = b0 < 0 ? 0 : (b0 > n_ids ? n_ids : b0);
        b1 = b1 < b0 ? b0 : (b1 > n_ids ? n_ids : b1);
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
        bool bad = false;
        for (int32_t j = b0; j < b1; ++j) {
            const int32_t id = ids[j];
            if (id < 0 || id >= n_blk) { bad = true; break; }
            const f32x4 b = pool4<BF>(B_pool, 4 * (((int64_t)id * H + h) * per_head4 + e));
            if (j == b0) {
                acc = b;
            } else {
                const float a = __expf(Lam[(int64_t)id * H + h]);
                acc = a * acc + b;
            }
            if (S_steps && j + 1 < b1) S_steps[((int64_t)(j - r) * H + h) * per_head4 + e] = acc;
        }
        if (bad) {
            const float f = __builtin_nanf("");
            acc = f32x4{f, f, f, f};
        }
        S[i] = acc;
    }
}

// ---------------------------------------------------------------- Mamba-2 block transitions
// Lambda = A_h * sum_t dt_t over each block (the scalar transition of Eq. 5):
// a segmented sum over the block's dt rows.  A workgroup covers 64 heads of
// one block with 16 token lanes (one wave each, so every load is one dt row
// segment of 256 bytes); each lane keeps several loads in flight, and the 16
// partial sums are added in a fixed order (reproducible results).
constexpr int LAM_LANES = 16;
__global__ __launch_bounds__(64 * LAM_LANES) void ssd_lambda_kernel(const int32_t* __restrict__ cu, int32_t n_seq,
                                                                    int64_t n_tok, int32_t H,
                                                                    const float* __restrict__ dt,
                                                                    const float* __restrict__ A,
                                                                    float* __restrict__ Lam) {
    __shared__ float part[LAM_LANES][64];
    const int hg = blockIdx.x % ((H + 63) / 64);
    const int s = blockIdx.x / ((H + 63) / 64);
    const int tl = threadIdx.x >> 6, hl = threadIdx.x & 63;
    const int h = hg * 64 + hl;
    int64_t t0 = cu[s], t1 = cu[s + 1];
    t0 = t0 < 0 ? 0 : (t0 > n_tok ? n_tok : t0);
    t1 = t1 < t0 ? t0 : (t1 > n_tok ? n_tok : t1);
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    if (h < H) {
        int64_t t = t0 + tl;
        for (; t + 3 * LAM_LANES < t1; t += 4 * LAM_LANES) {
#pragma unroll
            for (int u = 0; u < 4; ++u) acc[u] += dt[(t + u * LAM_LANES) * H + h];
        }
        for (; t < t1; t += LAM_LANES) acc[0] += dt[t * H + h];
    }
    part[tl][hl] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    __syncthreads();
    if (tl == 0 && h < H) {
        float sum = 0.f;
#pragma unroll
        for (int i = 0; i < LAM_LANES; ++i) sum += part[i][hl];
        Lam[(int64_t)s * H + h] = A[h] * sum;
    }
}

hipError_t launch_ssd_lambda(const int32_t* cu, int32_t n_seq, int64_t n_tok, int32_t H, const float* dt,
                             const float* A, float* Lam, hipStream_t st) {
    const int64_t grid = (int64_t)n_seq * ((H + 63) / 64);
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL(ssd_lambda_kernel, dim3((unsigned)grid), dim3(64 * LAM_LANES), 0, st, cu, n_seq, n_tok, H, dt,
                       A, Lam);
    return hipGetLastError();
}

hipError_t launch_compose_ssd(int32_t n_req, int32_t n_blk, int32_t H, int64_t per_head, const void* B_pool,
                              bool bf16_pool, const float* Lam, const int32_t* ids, const int32_t* blk_cu,
                              int32_t n_ids, float* S, float* S_steps, hipStream_t st) {
    const int64_t total = (int64_t)n_req * H * (per_head / 4);
    if (total == 0) return hipSuccess;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 256 * 16) blocks = 256 * 16;
    auto kern = bf16_pool ? compose_ssd_kernel<true> : compose_ssd_kernel<false>;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(256), 0, st, n_req, n_blk, H, per_head / 4, B_pool,
                       Lam, ids, blk_cu, n_ids, reinterpret_cast<f32x4*>(S), reinterpret_cast<f32x4*>(S_steps));
    return hipGetLastError();
}

// ---------------------------------------------------------------- Gated DeltaNet composition
// Work unit = (request, head, tile of 16*NW state rows); wave w owns rows
// row0 + 16w + (lane % 16).  The state stays in registers in acc-tile layout
// (tile nt: S[row][16nt + 4g + r]), which is directly the B operand of
//   S_new^T = M^T S^T    (contraction over the state's dk index),
// so each step stages only M in LDS (row-major, split into bf16 hi/lo planes;
// products Mh*Sh + Mh*Sl + Ml*Sh keep the fp32 chain at ~1e-5 relative) and
// reads the M^T fragments with transposed LDS loads.
//
// Software pipeline over the request's blocks: step j multiplies by M_j
// (staged in LDS one step earlier), then stages M_{j+1}, loaded one step
// earlier, and issues the loads of M_{j+2}; B_{j+1}'s rows are requested as
// soon as B_j has seeded the accumulators.  The two barriers of a step order
// LDS only (s_barrier after an LDS wait), so the global loads stay in flight
// across them, and nothing in the loop waits for every load in flight (see
// the block ids below).  Rows of a staged plane are DK + 16 elements apart,
// which keeps the transposed fragment reads free of bank conflicts; the LDS
// footprint (74 KB at dk = 128) lets two workgroups share a CU.  With S_steps,
// the state after each block but the request's last is also stored (request
// r's position j at row j - r).
//
// NW = 8 splits the state's dk tiles between two waves per row tile (wave w:
// row tile w % 4, dk half w / 4), each forming its half of S_new^T from half
// of M^T; the halves go through LDS (bf16 hi / lo, in each lane's acc-tile
// order) once per step, since every product needs the whole state.  A wave
// issues about one LDS read per 30 cycles whatever its width, and with four
// waves each reading all of M^T per step that issue time is the step's; the
// split halves the M^T reads per wave for 16 state reads more.
template <int DK>
struct ComposeLds {
    static constexpr int SM = DK >= 32 ? DK + 16 : DK + 8;
    static constexpr size_t PLANE = size_t(DK) * SM;  // elements
    static __host__ __device__ constexpr size_t bytes() { return 2 * PLANE * 2; }
    // the state halves of the eight-wave form: [4 row tiles][DK/16 tiles][hi, lo][64 lanes] x 4 bf16
    static __host__ __device__ constexpr size_t xbytes() { return size_t(4) * (DK / 16) * 2 * 64 * 8; }
};

template <int DK, int NW, bool BF>
__global__ __launch_bounds__(64 * NW) void compose_gdn_kernel(ComposeArgs p) {
    using Ly = ComposeLds<DK>;
    constexpr int NTK = DK / 16, SM = Ly::SM;
    constexpr bool CS = NW == 8;              // dk halves of the state on two waves per row tile
    static_assert(!CS || NTK % 2 == 0, "the eight-wave form needs dk >= 32");
    constexpr int NWR = CS ? 4 : NW;          // row tiles per workgroup
    constexpr int NOWN = CS ? NTK / 2 : NTK;  // dk tiles of the state a wave owns
    constexpr int NTH = 64 * NW;
    constexpr int NV = DK * DK / 4;              // float4 vectors of one M
    constexpr int PER = (NV + NTH - 1) / NTH;    // of them per thread
    // the matrix-core split needs every lane of the wave; it is used where each
    // thread stages whole vectors and the state chain is 32 wide.  The staging
    // of M uses it with four waves only: a smaller workgroup stages M with as
    // many split products per wave as it has state products, and that wave's
    // matrix-core time becomes the step's
    constexpr bool MM_SPLIT = NV % NTH == 0 && NTK % 2 == 0;
    constexpr bool MM_SPLIT_M = MM_SPLIT && NW >= 4;
    extern __shared__ __align__(16) char smem[];
    bf16* sMh = reinterpret_cast<bf16*>(smem);
    bf16* sMl = sMh + Ly::PLANE;
    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, g = lane >> 4, c16 = lane & 15;
    const int rt = CS ? (w & 3) : w;        // row tile
    const int nt0 = CS ? (w >> 2) * NOWN : 0;  // first dk tile of the state this wave owns
    const bf16x8 negI = neg_eye(g, c16);
    // the state halves (eight-wave form): slot of dk tile nt, plane pl of this row tile
    auto sx = [&](int nt, int pl) {
        return reinterpret_cast<bf16x4*>(smem + Ly::bytes()) + ((rt * NTK + nt) * 2 + pl) * 64 + lane;
    };
    // units: the row tiles of one (request, head) adjacent, then the request
    // index fastest, so each XCD's range holds a few heads of every request
    // (ragged block counts load the XCDs evenly)
    const int u = xcd_unit(blockIdx.x, p.n_units);
    const int n_req = p.n_units / (p.tiles * p.h_v);
    const int tile = u % p.tiles;
    const int r = (u / p.tiles) % n_req;
    const int h = u / (p.tiles * n_req);
    const int my_row = tile * 16 * NWR + 16 * rt + c16;

    int32_t b0 = p.blk_cu[r], b1 = p.blk_cu[r + 1];
    b0 = b0 < 0 ? 0 : (b0 > p.n_ids ? p.n_ids : b0);
    b1 = b1 < b0 ? b0 : (b1 > p.n_ids ? p.n_ids : b1);

    auto valid = [&](int32_t id) { return id >= 0 && id < p.n_blk; };
    auto b_rows = [&](int32_t id) {  // element offset of this lane's B row segment
        return (((int64_t)id * p.h_v + h) * p.dv + my_row) * DK + 16 * nt0 + 4 * g;
    };
    f32x4 mreg[PER], breg[NOWN];
    auto load_m = [&](int32_t id) {
        // plain loads: the head's other row tiles read the same M through the XCD's L2
        const f32x4* Mj = reinterpret_cast<const f32x4*>(p.M_pool + ((int64_t)id * p.h_v + h) * DK * DK);
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * NTH;
            if (NV % NTH == 0 || idx < NV) mreg[i] = Mj[idx];
        }
    };
    auto load_b = [&](int32_t id) {
        const int64_t Bj = b_rows(id);
#pragma unroll
        for (int nt = 0; nt < NOWN; ++nt) breg[nt] = pool4<BF>(p.B_pool, Bj + 16 * nt);
    };
    // M (in mreg) -> bf16 hi / lo planes in LDS, row-major
    auto stage_m = [&]() {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * NTH;
            if (NV % NTH != 0 && idx >= NV) continue;
            const int ii = idx / (DK / 4), jj = (idx % (DK / 4)) * 4;
            const Split4 sp = MM_SPLIT_M ? split4_mm(mreg[i], negI) : split4(mreg[i]);
            *reinterpret_cast<bf16x4*>(sMh + ii * SM + jj) = sp.hi;
            *reinterpret_cast<bf16x4*>(sMl + ii * SM + jj) = sp.lo;
        }
    };

    // The request's block ids are read through the scalar cache (a constant
    // address-space view of the read-only id array): their waits count on the
    // scalar/LDS counter, so reading an id never waits for the prefetched M and
    // B loads in flight on the vector-memory counter.
    typedef __attribute__((address_space(4))) const int32_t const_i32;
    const const_i32* ids_c = (const const_i32*)p.blk_ids;
    auto id_at = [&](int32_t j) { return ids_c[j]; };
    f32x4 S[NOWN];
#pragma unroll
    for (int nt = 0; nt < NOWN; ++nt) S[nt] = zero4();
    // block ids are the same for every wave of the workgroup, so every branch
    // on them below is uniform; bad_at is the first position with an invalid id
    int32_t bad_at = b1;
    auto id_checked = [&](int32_t j) {
        const int32_t id = id_at(j);
        if (!valid(id) && j < bad_at) bad_at = j;
        return id;
    };
    // Step j (b0 <= j < b1) starts with B_j in breg, M_{j+1} in mreg and, past
    // the first step, M_j staged in LDS; it seeds the accumulators
    // with B_j, requests B_{j+1}, adds M_j^T S^T (not on the first step, which
    // only takes S = B_{b0}), stages M_{j+1} and requests M_{j+2}.  Every step
    // has the same shape, so the state never comes straight from a load and
    // the prefetch registers carry the same in-flight loads at the top of
    // every step.  Loads past the request's end or its first invalid id
    // re-read the last valid block (a cache hit; unconditional loads keep the
    // prefetch registers single-valued).
    int32_t id0 = 0, id1 = 0, id2 = 0;  // ids at positions j, j + 1, j + 2
    if (b0 < b1) id0 = id_checked(b0);
    if (b0 + 1 < b1) id1 = id_checked(b0 + 1);
    if (b0 < bad_at) {
        load_b(id0);
        load_m(b0 + 1 < bad_at ? id1 : id0);
    }
    for (int32_t j = b0; j < b1 && j < bad_at; ++j) {
        if (j + 2 < b1) id2 = id_checked(j + 2);
        lds_barrier();  // M_j staged by every wave (eight waves: and the state halves published)
        f32x4 acc[NOWN];
#pragma unroll
        for (int nt = 0; nt < NOWN; ++nt) acc[nt] = breg[nt];
        load_b(j + 1 < bad_at ? id1 : id0);
        // B_{j+1} stays ahead of M_{j+2} in issue order: the memory counter is
        // in order, so waiting for one waits for everything issued before it
        __builtin_amdgcn_sched_barrier(0);
        if (j > b0) {
            bf16x4 Sh[NTK], Sl[NTK];
            if constexpr (CS) {
                // the whole state, both halves as published after the previous step
#pragma unroll
                for (int nt = 0; nt < NTK; ++nt) {
                    Sh[nt] = *sx(nt, 0);
                    Sl[nt] = *sx(nt, 1);
                }
            } else {
#pragma unroll
                for (int nt = 0; nt < NTK; ++nt) {
                    const Split4 sp = MM_SPLIT ? split4_mm(S[nt], negI) : split4(S[nt]);
                    Sh[nt] = sp.hi;
                    Sl[nt] = sp.lo;
                }
            }
            // S_new^T tile nt (rows 16nt..16nt+15) = M^T S^T + B^T: A fragments of
            // M^T come straight from the row-major planes through transposed LDS
            // reads; the dk tiles are interleaved so NTK accumulation chains are in
            // flight
            if constexpr (NTK == 1) {
                const bf16x4 a0 = lds4_tr(sMh, SM, 0, 0, g, c16);
                const bf16x4 c0 = lds4_tr(sMl, SM, 0, 0, g, c16);
                acc[0] = mma16(a0, Sh[0], acc[0]);
                acc[0] = mma16(a0, Sl[0], acc[0]);
                acc[0] = mma16(c0, Sh[0], acc[0]);
            } else {
#pragma unroll
                for (int kg = 0; kg < NTK; kg += 2) {
                    bf16x4 a0[NOWN], a1[NOWN], c0[NOWN], c1[NOWN];
#pragma unroll
                    for (int nt = 0; nt < NOWN; ++nt) {
                        a0[nt] = lds4_tr(sMh, SM, 16 * kg, 16 * (nt0 + nt), g, c16);
                        a1[nt] = lds4_tr(sMh, SM, 16 * kg + 16, 16 * (nt0 + nt), g, c16);
                        c0[nt] = lds4_tr(sMl, SM, 16 * kg, 16 * (nt0 + nt), g, c16);
                        c1[nt] = lds4_tr(sMl, SM, 16 * kg + 16, 16 * (nt0 + nt), g, c16);
                    }
#pragma unroll
                    for (int nt = 0; nt < NOWN; ++nt) {
                        acc[nt] = mma32(a0[nt], a1[nt], Sh[kg], Sh[kg + 1], acc[nt]);
                        acc[nt] = mma32(a0[nt], a1[nt], Sl[kg], Sl[kg + 1], acc[nt]);
                        acc[nt] = mma32(c0[nt], c1[nt], Sh[kg], Sh[kg + 1], acc[nt]);
                    }
                }
            }
        }
        // stage M_{j+1} (requested one step ago) and request M_{j+2}
        lds_barrier();  // every wave is done reading M_j (and the state halves)
        stage_m();
        load_m(j + 2 < bad_at ? id2 : (j + 1 < bad_at ? id1 : id0));
#pragma unroll
        for (int nt = 0; nt < NOWN; ++nt) S[nt] = acc[nt];
        if constexpr (CS) {
            // this wave's half of the new state, split, for every wave of its row tile
#pragma unroll
            for (int nt = 0; nt < NOWN; ++nt) {
                const Split4 sp = split4_mm(acc[nt], negI);
                *sx(nt0 + nt, 0) = sp.hi;
                *sx(nt0 + nt, 1) = sp.lo;
            }
        }
        if (p.S_steps && j + 1 < b1) {
            // the state after this block (position j), a start state for a later step
            float* dst = p.S_steps + ((((int64_t)j - r) * p.h_v + h) * p.dv + my_row) * DK + 16 * nt0 + 4 * g;
#pragma unroll
            for (int nt = 0; nt < NOWN; ++nt) *reinterpret_cast<f32x4*>(dst + 16 * nt) = acc[nt];
        }
        id0 = id1;
        id1 = id2;
    }
    if (bad_at < b1) {
        const float f = __builtin_nanf("");
#pragma unroll
        for (int nt = 0; nt < NOWN; ++nt) S[nt] = f32x4{f, f, f, f};
    }
    float* dst = p.S + (((int64_t)r * p.h_v + h) * p.dv + my_row) * DK + 16 * nt0 + 4 * g;
#pragma unroll
    for (int nt = 0; nt < NOWN; ++nt) *reinterpret_cast<f32x4*>(dst + 16 * nt) = S[nt];
}

template <int DK, int NW>
static hipError_t launch_compose_gdn_nw(const ComposeArgs& a, hipStream_t st) {
    const size_t lds = ComposeLds<DK>::bytes() + (NW == 8 ? ComposeLds<DK>::xbytes() : 0);
    auto kern = a.bf16_pool ? compose_gdn_kernel<DK, NW, true> : compose_gdn_kernel<DK, NW, false>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3(a.n_units), dim3(64 * NW), lds, st, a);
    return hipGetLastError();
}

template <int DK>
static hipError_t launch_compose_gdn_t(const ComposeArgs& a, hipStream_t st) {
    switch (a.nw) {
        case 1: return launch_compose_gdn_nw<DK, 1>(a, st);
        case 2: return launch_compose_gdn_nw<DK, 2>(a, st);
        case 4: return launch_compose_gdn_nw<DK, 4>(a, st);
        case 8:
            if constexpr (DK >= 32) return launch_compose_gdn_nw<DK, 8>(a, st);
            return hipErrorInvalidValue;
    }
    return hipErrorInvalidValue;
}

hipError_t launch_compose_gdn(int dk, const ComposeArgs& a, hipStream_t st) {
    switch (dk) {
        case 16: return launch_compose_gdn_t<16>(a, st);
        case 32: return launch_compose_gdn_t<32>(a, st);
        case 64: return launch_compose_gdn_t<64>(a, st);
        case 128: return launch_compose_gdn_t<128>(a, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace lkv
