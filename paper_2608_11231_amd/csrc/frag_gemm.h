// Fragment-level matrix-core products used by the chunk kernel, and the
// register prefetch of token tiles.  Conventions (acc tiles, the contraction
// index bijection, the transposed LDS read) are described in lkv_device.h.
#pragma once
#include <type_traits>

#include "lkv_device.h"

namespace lkv {

// Multi-tile products with interleaved accumulation chains.  One MFMA chain
// per output tile serialises on the matrix-core latency; looping over the
// contraction slices outside and the tiles inside keeps NM independent chains
// in flight.  nk = number of 16-slices (1, or even).

// acc[m] += A_m x B (all passes), for NM tiles whose A rows are LDS rows
// `a0 + m * mstep` of a K / Q tile in kq_pos order (this lane's row, hi plane;
// lo plane at + plane), B = acc-layout register tiles (hi bh, lo bl).  Within
// each contraction slice the passes are issued pass-major (every tile's hi pass,
// then every tile's lo passes), so consecutive products never share an
// accumulator.
template <int NM, bool ALO, bool BLO>
__device__ __forceinline__ void mgemm_rows(const bf16* a0, int mstep, int plane, const bf16x4* bh,
                                           const bf16x4* bl, int nk, int g, f32x4* acc) {
    if (nk == 1) {
#pragma unroll
        for (int m = 0; m < NM; ++m) {
            const bf16* ar = a0 + m * mstep + 4 * g;
            const bf16x4 x = lds4(ar);
            acc[m] = mma16(x, bh[0], acc[m]);
            if (BLO) acc[m] = mma16(x, bl[0], acc[m]);
            if (ALO) acc[m] = mma16(lds4(ar + plane), bh[0], acc[m]);
        }
        return;
    }
    // every fragment is requested before the first product, so the LDS latency is
    // paid once rather than once per product
    constexpr int NP = 4;  // 32-wide slices, at most 128 / 32
    bf16x8 xh[NP][NM], xl[ALO ? NP : 1][NM];
#pragma unroll
    for (int kp = 0; kp < NP; ++kp) {
        if (2 * kp >= nk) break;
#pragma unroll
        for (int m = 0; m < NM; ++m) {
            const bf16* ar = a0 + m * mstep + 32 * kp + 8 * g;
            xh[kp][m] = lds8(ar);
            if constexpr (ALO) xl[kp][m] = lds8(ar + plane);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kp = 0; kp < NP; ++kp) {
        if (2 * kp >= nk) break;
#pragma unroll
        for (int m = 0; m < NM; ++m) acc[m] = mma32(xh[kp][m], bh[2 * kp], bh[2 * kp + 1], acc[m]);
        if (BLO) {
#pragma unroll
            for (int m = 0; m < NM; ++m) acc[m] = mma32(xh[kp][m], bl[2 * kp], bl[2 * kp + 1], acc[m]);
        }
        if constexpr (ALO) {
#pragma unroll
            for (int m = 0; m < NM; ++m) acc[m] = mma32(xl[kp][m], bh[2 * kp], bh[2 * kp + 1], acc[m]);
        }
    }
}

// mgemm_rows for RT independent right-hand sides B_rt (the state row tiles of
// one wave) sharing every A fragment: acc[rt][m] += A_m x B_rt (all passes,
// pass-major).  nk = NTK 16-slices (even, at least 2).
template <int NM, int RT, int NTK, bool ALO, bool BLO>
__device__ __forceinline__ void mgemm_rows_rt(const bf16* a0, int mstep, int plane, const bf16x4 (&bh)[RT][NTK],
                                              const bf16x4 (&bl)[RT][NTK], int g, f32x4 (&acc)[RT][NM]) {
    static_assert(NTK % 2 == 0, "32-wide slices");
    constexpr int NP = NTK / 2;
#pragma unroll
    for (int kp = 0; kp < NP; ++kp) {
        bf16x8 xh[NM], xl[ALO ? NM : 1];
#pragma unroll
        for (int m = 0; m < NM; ++m) {
            const bf16* ar = a0 + m * mstep + 32 * kp + 8 * g;
            xh[m] = lds8(ar);
            if constexpr (ALO) xl[m] = lds8(ar + plane);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int m = 0; m < NM; ++m)
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
                acc[rt][m] = mma32(xh[m], bh[rt][2 * kp], bh[rt][2 * kp + 1], acc[rt][m]);
        if (BLO) {
#pragma unroll
            for (int m = 0; m < NM; ++m)
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
                    acc[rt][m] = mma32(xh[m], bl[rt][2 * kp], bl[rt][2 * kp + 1], acc[rt][m]);
        }
        if constexpr (ALO) {
#pragma unroll
            for (int m = 0; m < NM; ++m)
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
                    acc[rt][m] = mma32(xl[m], bh[rt][2 * kp], bh[rt][2 * kp + 1], acc[rt][m]);
        }
    }
}

// mgemm_tr for RT right-hand sides sharing every transposed A fragment:
// acc[rt][n] += M^T(columns 16n..) x B_rt, nk = NK token 16-slices (even).
template <int DK, int NN, int RT, int NK, bool ALO, bool BLO>
__device__ __forceinline__ void mgemm_tr_rt(const bf16* M, int plane, int stride, const bf16x4 (&bh)[RT][NK],
                                            const bf16x4 (&bl)[RT][NK], int g, int c, f32x4 (&acc)[RT][NN]) {
    static_assert(NK % 2 == 0, "32-wide slices");
#pragma unroll
    for (int kg = 0; kg < NK; kg += 2) {
        bf16x4 x0[NN], x1[NN], y0[ALO ? NN : 1], y1[ALO ? NN : 1];
#pragma unroll
        for (int n = 0; n < NN; ++n) {
            x0[n] = lds4_tr_kq<DK>(M, stride, 16 * kg, 16 * n, g, c);
            x1[n] = lds4_tr_kq<DK>(M, stride, 16 * kg + 16, 16 * n, g, c);
            if constexpr (ALO) {
                y0[n] = lds4_tr_kq<DK>(M + plane, stride, 16 * kg, 16 * n, g, c);
                y1[n] = lds4_tr_kq<DK>(M + plane, stride, 16 * kg + 16, 16 * n, g, c);
            }
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int n = 0; n < NN; ++n)
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                acc[rt][n] = mma32(x0[n], x1[n], bh[rt][kg], bh[rt][kg + 1], acc[rt][n]);
                if (BLO) acc[rt][n] = mma32(x0[n], x1[n], bl[rt][kg], bl[rt][kg + 1], acc[rt][n]);
                if constexpr (ALO) acc[rt][n] = mma32(y0[n], y1[n], bh[rt][kg], bh[rt][kg + 1], acc[rt][n]);
            }
    }
}

// acc[n] += M^T(columns 16n..16n+15) x B for NN tiles, the A fragments read
// transposed from a token-major K / Q tile M in kq_pos<DK> order (rows =
// contraction, hi plane; lo plane at + plane).  All passes accumulate into acc[n].
template <int DK, int NN, bool ALO, bool BLO>
__device__ __forceinline__ void mgemm_tr(const bf16* M, int plane, int stride, const bf16x4* bh, const bf16x4* bl,
                                         int nk, int g, int c, f32x4* acc) {
    if (nk == 1) {
#pragma unroll
        for (int n = 0; n < NN; ++n) {
            const bf16x4 x = lds4_tr_kq<DK>(M, stride, 0, 16 * n, g, c);
            acc[n] = mma16(x, bh[0], acc[n]);
            if (BLO) acc[n] = mma16(x, bl[0], acc[n]);
            if (ALO) acc[n] = mma16(lds4_tr_kq<DK>(M + plane, stride, 0, 16 * n, g, c), bh[0], acc[n]);
        }
        return;
    }
    // fragments of one pair of contraction slices are all requested before its products
#pragma unroll
    for (int kg = 0; kg < 8; kg += 2) {
        if (kg >= nk) break;
        bf16x4 x0[NN], x1[NN], y0[ALO ? NN : 1], y1[ALO ? NN : 1];
#pragma unroll
        for (int n = 0; n < NN; ++n) {
            x0[n] = lds4_tr_kq<DK>(M, stride, 16 * kg, 16 * n, g, c);
            x1[n] = lds4_tr_kq<DK>(M, stride, 16 * kg + 16, 16 * n, g, c);
            if constexpr (ALO) {
                y0[n] = lds4_tr_kq<DK>(M + plane, stride, 16 * kg, 16 * n, g, c);
                y1[n] = lds4_tr_kq<DK>(M + plane, stride, 16 * kg + 16, 16 * n, g, c);
            }
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int n = 0; n < NN; ++n) {
            acc[n] = mma32(x0[n], x1[n], bh[kg], bh[kg + 1], acc[n]);
            if (BLO) acc[n] = mma32(x0[n], x1[n], bl[kg], bl[kg + 1], acc[n]);
            if constexpr (ALO) acc[n] = mma32(y0[n], y1[n], bh[kg], bh[kg + 1], acc[n]);
        }
    }
}

// Store an acc tile (rows 4g+r, column c) TRANSPOSED into a 16x16 block:
// XT[c][4g + r] = v[r] (hi, and lo plane at `plane` when LO); one 8-byte write
// per lane and plane.
//
// The stores stay where they are written (compiler memory barrier): the kernels
// call this from branches on the wave index, and letting the optimizer sink the
// stores of several branches into one shared store after the branches has been
// seen to produce wrong data in LDS.
template <int SB, bool LO>
__device__ __forceinline__ void store_tile_tr(bf16* XT, int plane, f32x4 v, int g, int c) {
    if (LO) {
        const Split4 sp = split4(v);
        *reinterpret_cast<bf16x4*>(XT + c * SB + 4 * g) = sp.hi;
        *reinterpret_cast<bf16x4*>(XT + plane + c * SB + 4 * g) = sp.lo;
    } else {
        *reinterpret_cast<bf16x4*>(XT + c * SB + 4 * g) = to_bf16(v);
    }
    asm volatile("" ::: "memory");
}

// A [CH x DK] token-major K / Q tile prefetched into registers and committed
// to LDS in kq_pos<DK> order.  Each thread handles units of 8 consecutive
// source columns of one row, fetched from global memory as one 16-byte load
// (two for fp32 inputs, which are split into bf16 hi / lo planes at commit);
// the unit's two aligned 4-column runs land at their kq_pos places as two
// 8-byte LDS writes per plane.  Rows t >= n read as zero.
// Raw buffer resource over [base, base + bytes): 16-byte loads at offsets at or
// past the end return zeros (the hardware range check), so tile tails need no
// branches.  Word 3 is the untyped-access configuration of gfx9-family parts.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint32_t buf_load4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
__device__ __forceinline__ uint32_t buf_load2(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}
__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
    const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
    return uint4{v[0], v[1], v[2], v[3]};
}

template <int CH, int DK, bool F32IO, int NTH>
struct KQTile {
    static constexpr int UPR = DK / 8;                // units per row
    static constexpr int NU = CH * UPR;               // units per tile
    static constexpr int PER = (NU + NTH - 1) / NTH;  // units per thread
    static constexpr int ES = F32IO ? 4 : 2;          // element bytes in global memory
    uint4 a[PER], b[F32IO ? PER : 1];                 // bf16: 8 columns; fp32: columns 0-3 / 4-7

    __device__ __forceinline__ void load(const char* base, uint32_t row_bytes, int n, int tid) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * NTH;
            const int t = idx / UPR, u = idx % UPR;
            uint4 x{}, y{};
            if (idx < NU && t < n) {
                const char* src = base + (uint32_t)t * row_bytes + ES * 8 * u;
                x = *reinterpret_cast<const uint4*>(src);
                if constexpr (F32IO) y = *reinterpret_cast<const uint4*>(src + 16);
            }
            a[i] = x;
            if constexpr (F32IO) b[i] = y;
        }
    }
    // The same through a buffer resource whose range ends at the segment's end:
    // rows past it (and units past the tile) read as zero without a branch.
    // chunk_off = byte offset of the chunk's first row from the resource base.
    __device__ __forceinline__ void load_buf(__amdgpu_buffer_rsrc_t r, uint32_t chunk_off, uint32_t row_bytes,
                                             int tid) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * NTH;
            const int t = idx / UPR, u = idx % UPR;
            const uint32_t off = (NU % NTH != 0 && idx >= NU) ? 0xffffffffu
                                                                : chunk_off + (uint32_t)t * row_bytes + ES * 8 * u;
            a[i] = buf_load16(r, off);
            if constexpr (F32IO) b[i] = buf_load16(r, off == 0xffffffffu ? off : off + 16);
        }
    }
    // units to LDS rows of stride ds elements (lo plane at dst + pofs for fp32 io)
    __device__ __forceinline__ void commit(bf16* dst, int ds, int pofs, int tid) const {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * NTH;
            if (NU % NTH != 0 && idx >= NU) continue;
            const int t = idx / UPR, u = idx % UPR;
            bf16* d = dst + t * ds;
            const int p0 = kq_pos<DK>(8 * u), p1 = kq_pos<DK>(8 * u + 4);
            if constexpr (!F32IO) {
                *reinterpret_cast<uint2*>(d + p0) = uint2{a[i].x, a[i].y};
                *reinterpret_cast<uint2*>(d + p1) = uint2{a[i].z, a[i].w};
            } else {
                const Split4 sa = split4(__builtin_bit_cast(f32x4, a[i]));
                const Split4 sb = split4(__builtin_bit_cast(f32x4, b[i]));
                *reinterpret_cast<bf16x4*>(d + p0) = sa.hi;
                *reinterpret_cast<bf16x4*>(d + p1) = sb.hi;
                *reinterpret_cast<bf16x4*>(d + pofs + p0) = sa.lo;
                *reinterpret_cast<bf16x4*>(d + pofs + p1) = sb.lo;
            }
        }
    }
};

// A [CH x NCOL] token-major tile of a global tensor, prefetched into registers
// (16-byte vectors spread over NTH threads) and later committed to LDS
// row-major.  Rows t >= n read as zero.
template <int CH, int NCOL, bool F32IO, int NTH>
struct TileRegs {
    static constexpr int EPV = F32IO ? 4 : 8;        // elements per 16-byte vector
    static constexpr int VPR = NCOL / EPV;            // vectors per row
    static constexpr int NV = CH * VPR;               // vectors per tile
    static constexpr int PER = (NV + NTH - 1) / NTH;  // vectors per thread
    uint4 r[PER];

    // element (t, c) of the source lives at base + t*row_bytes + c*sizeof(elem):
    // a wave-uniform 64-bit base plus a 32-bit per-lane byte offset
    __device__ __forceinline__ void load(const char* base, uint32_t row_bytes, int n, int tid) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * NTH;
            const int t = idx / VPR, cv = idx % VPR;
            uint4 x = uint4{0u, 0u, 0u, 0u};
            if (idx < NV && t < n) x = *reinterpret_cast<const uint4*>(base + (uint32_t)t * row_bytes + 16u * cv);
            r[i] = x;
        }
    }
    // through a buffer resource ending at the segment's end (see KQTile::load_buf)
    __device__ __forceinline__ void load_buf(__amdgpu_buffer_rsrc_t rs, uint32_t chunk_off, uint32_t row_bytes,
                                             int tid) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * NTH;
            const int t = idx / VPR, cv = idx % VPR;
            r[i] = buf_load16(rs, idx < NV ? chunk_off + (uint32_t)t * row_bytes + 16u * cv : 0xffffffffu);
        }
    }
    // row-major into dst (row stride ds elements; lo plane at dst + pofs for fp32 io)
    __device__ __forceinline__ void commit(bf16* dst, int ds, int pofs, int tid) const {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * NTH;
            if (idx >= NV) continue;
            const int t = idx / VPR, c = (idx % VPR) * EPV;
            if (!F32IO) {
                *reinterpret_cast<uint4*>(dst + t * ds + c) = r[i];
            } else {
                const Split4 sp = split4(__builtin_bit_cast(f32x4, r[i]));
                *reinterpret_cast<bf16x4*>(dst + t * ds + c) = sp.hi;
                *reinterpret_cast<bf16x4*>(dst + pofs + t * ds + c) = sp.lo;
            }
        }
    }
};

}  // namespace lkv
