// Fragment-level matrix-core products used by the chunk kernel, and the
// register prefetch of token tiles.  Conventions (acc tiles, the contraction
// index bijection, the transposed LDS read) are described in lkv_device.h.
#pragma once
#include "lkv_device.h"

namespace lkv {

// acc += A x B over 16-slices [kb, ke) of the contraction index.
//   A: row-major LDS rows (ah: the lane's row in the hi plane, al_: lo plane);
//      slice kg covers elements 16kg..16kg+15 of the row.
//   B: acc-layout register tiles bh[kg] / bl[kg] (hi / lo).
// Passes: hi*hi, plus hi*lo when BLO, plus lo*hi when ALO.  Pairs of slices go
// through the 32-wide MFMA; an odd tail after pairs is zero-padded so that one
// accumulation chain never mixes MFMA shapes.
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
        if (kg == kb) {
            acc = mma16(a0, bh[kg], acc);
            if (BLO) acc = mma16(a0, bl[kg], acc);
            if (ALO) acc = mma16(lds4(al_ + 16 * kg + 4 * g), bh[kg], acc);
        } else {
            const bf16x4 z = zero_bf16x4();
            acc = mma32(a0, z, bh[kg], z, acc);
            if (BLO) acc = mma32(a0, z, bl[kg], z, acc);
            if (ALO) acc = mma32(lds4(al_ + 16 * kg + 4 * g), z, bh[kg], z, acc);
        }
    }
    return acc;
}

// acc += A x B with A = M^T: the A fragments of slice kg are rows 16kg.. of a
// row-major LDS matrix M (planes Mh / Ml, row stride `stride`), columns
// c0..c0+15, read with transposed LDS loads.  B as in gemm_lds_reg.
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

// acc += sum over slices kg in [kb, ke) of X_kg x B[kg], where each 16x16 block
// X_kg is stored TRANSPOSED (XT[i][t] = X[t][i], row stride SB) at blk(kg) in
// hi / lo planes (lo at blk(kg) + plane).  All passes (hi*hi, hi*lo, lo*hi).
template <int SB, bool ALO, bool BLO, typename BlkFn>
__device__ __forceinline__ f32x4 gemm_blk_reg(BlkFn blk, int plane, const bf16x4* bh, const bf16x4* bl, int kb,
                                              int ke, int g, int c, f32x4 acc) {
    int kg = kb;
    for (; kg + 1 < ke; kg += 2) {
        const bf16* x0 = blk(kg);
        const bf16* x1 = blk(kg + 1);
        const bf16x4 a0 = lds4_tr(x0, SB, 0, 0, g, c), a1 = lds4_tr(x1, SB, 0, 0, g, c);
        acc = mma32(a0, a1, bh[kg], bh[kg + 1], acc);
        if (BLO) acc = mma32(a0, a1, bl[kg], bl[kg + 1], acc);
        if (ALO) {
            const bf16x4 c0 = lds4_tr(x0 + plane, SB, 0, 0, g, c), c1 = lds4_tr(x1 + plane, SB, 0, 0, g, c);
            acc = mma32(c0, c1, bh[kg], bh[kg + 1], acc);
        }
    }
    if (kg < ke) {
        const bf16* x0 = blk(kg);
        const bf16x4 a0 = lds4_tr(x0, SB, 0, 0, g, c);
        if (kg == kb) {
            acc = mma16(a0, bh[kg], acc);
            if (BLO) acc = mma16(a0, bl[kg], acc);
            if (ALO) acc = mma16(lds4_tr(x0 + plane, SB, 0, 0, g, c), bh[kg], acc);
        } else {
            const bf16x4 z = zero_bf16x4();
            acc = mma32(a0, z, bh[kg], z, acc);
            if (BLO) acc = mma32(a0, z, bl[kg], z, acc);
            if (ALO) acc = mma32(lds4_tr(x0 + plane, SB, 0, 0, g, c), z, bh[kg], z, acc);
        }
    }
    return acc;
}

// Multi-tile products with interleaved accumulation chains.  One MFMA chain
// per output tile serialises on the matrix-core latency; looping over the
// contraction slices outside and the tiles inside keeps NM independent chains
// in flight.  nk = number of 16-slices (1, or even).

// acc_h[m] += A_m x B (hi passes), acc_l[m] += lo passes, for NM tiles whose A
// rows are LDS rows `a0 + m * mstep` (this lane's row, hi plane; lo plane at
// + plane), B = acc-layout register tiles.
template <int NM, bool ALO, bool BLO>
__device__ __forceinline__ void mgemm_rows(const bf16* a0, int mstep, int plane, const bf16x4* bh,
                                           const bf16x4* bl, int nk, int g, f32x4* acc_h, f32x4* acc_l) {
    if (nk == 1) {
#pragma unroll
        for (int m = 0; m < NM; ++m) {
            const bf16* ar = a0 + m * mstep + 4 * g;
            const bf16x4 x = lds4(ar);
            acc_h[m] = mma16(x, bh[0], acc_h[m]);
            if (BLO) acc_l[m] = mma16(x, bl[0], acc_l[m]);
            if (ALO) acc_l[m] = mma16(lds4(ar + plane), bh[0], acc_l[m]);
        }
        return;
    }
#pragma unroll
    for (int kg = 0; kg < 8; kg += 2) {
        if (kg >= nk) break;
#pragma unroll
        for (int m = 0; m < NM; ++m) {
            const bf16* ar = a0 + m * mstep + 16 * kg + 4 * g;
            const bf16x4 x0 = lds4(ar), x1 = lds4(ar + 16);
            acc_h[m] = mma32(x0, x1, bh[kg], bh[kg + 1], acc_h[m]);
            if (BLO) acc_l[m] = mma32(x0, x1, bl[kg], bl[kg + 1], acc_l[m]);
            if (ALO) acc_l[m] = mma32(lds4(ar + plane), lds4(ar + plane + 16), bh[kg], bh[kg + 1], acc_l[m]);
        }
    }
}

// acc[n] += M^T(columns 16n..16n+15) x B for NN tiles, the A fragments read
// transposed from a row-major LDS matrix M (rows = contraction, hi plane; lo
// plane at + plane).  All passes accumulate into acc[n].
template <int NN, bool ALO, bool BLO>
__device__ __forceinline__ void mgemm_tr(const bf16* M, int plane, int stride, const bf16x4* bh, const bf16x4* bl,
                                         int nk, int g, int c, f32x4* acc) {
    if (nk == 1) {
#pragma unroll
        for (int n = 0; n < NN; ++n) {
            const bf16x4 x = lds4_tr(M, stride, 0, 16 * n, g, c);
            acc[n] = mma16(x, bh[0], acc[n]);
            if (BLO) acc[n] = mma16(x, bl[0], acc[n]);
            if (ALO) acc[n] = mma16(lds4_tr(M + plane, stride, 0, 16 * n, g, c), bh[0], acc[n]);
        }
        return;
    }
#pragma unroll
    for (int kg = 0; kg < 8; kg += 2) {
        if (kg >= nk) break;
#pragma unroll
        for (int n = 0; n < NN; ++n) {
            const bf16x4 x0 = lds4_tr(M, stride, 16 * kg, 16 * n, g, c);
            const bf16x4 x1 = lds4_tr(M, stride, 16 * kg + 16, 16 * n, g, c);
            acc[n] = mma32(x0, x1, bh[kg], bh[kg + 1], acc[n]);
            if (BLO) acc[n] = mma32(x0, x1, bl[kg], bl[kg + 1], acc[n]);
            if (ALO) {
                const bf16x4 y0 = lds4_tr(M + plane, stride, 16 * kg, 16 * n, g, c);
                const bf16x4 y1 = lds4_tr(M + plane, stride, 16 * kg + 16, 16 * n, g, c);
                acc[n] = mma32(y0, y1, bh[kg], bh[kg + 1], acc[n]);
            }
        }
    }
}

// acc += A(LDS rows) x B(LDS rows)^T over DK, both read with the same pattern.
template <int DK, bool LO>
__device__ __forceinline__ f32x4 gemm_lds_lds(const bf16* ah, const bf16* al_, const bf16* bh, const bf16* bl,
                                              int g, f32x4 acc) {
    constexpr int NK = DK / 16;
    if (NK == 1) {
        const int o0 = 4 * g;
        const bf16x4 a0 = lds4(ah + o0), b0 = lds4(bh + o0);
        acc = mma16(a0, b0, acc);
        if (LO) {
            acc = mma16(a0, lds4(bl + o0), acc);
            acc = mma16(lds4(al_ + o0), b0, acc);
        }
        return acc;
    }
    // even and odd slice pairs accumulate separately: two chains in flight
    f32x4 acc2 = zero4();
#pragma unroll
    for (int kg = 0; kg + 1 < NK; kg += 2) {
        const int o0 = 16 * kg + 4 * g, o1 = o0 + 16;
        const bf16x4 a0 = lds4(ah + o0), a1 = lds4(ah + o1), b0 = lds4(bh + o0), b1 = lds4(bh + o1);
        f32x4& t = ((kg >> 1) & 1) ? acc2 : acc;
        t = mma32(a0, a1, b0, b1, t);
        if (LO) {
            t = mma32(a0, a1, lds4(bl + o0), lds4(bl + o1), t);
            t = mma32(lds4(al_ + o0), lds4(al_ + o1), b0, b1, t);
        }
    }
    return acc + acc2;
}

// Store an acc tile (rows 4g+r, column c) TRANSPOSED into a 16x16 block:
// XT[c][4g + r] = v[r] (hi, and lo plane at `plane` when LO); one 8-byte write
// per lane and plane.
template <int SB, bool LO>
__device__ __forceinline__ void store_tile_tr(bf16* XT, int plane, f32x4 v, int g, int c) {
    if (LO) {
        const Split4 sp = split4(v);
        *reinterpret_cast<bf16x4*>(XT + c * SB + 4 * g) = sp.hi;
        *reinterpret_cast<bf16x4*>(XT + plane + c * SB + 4 * g) = sp.lo;
    } else {
        *reinterpret_cast<bf16x4*>(XT + c * SB + 4 * g) = to_bf16(v);
    }
}

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
