// Child scoring on the matrix cores (§2.2 child-scoring equation), shared by
// the encoder (activations x) and the decode-backward (upstream gradient g).
//
// For level l, a block of 16 columns r = tt*CPT + q (token tt, parent slot q)
// with parent index p_r, and a tile of 16 generators j:
//     S[j][r] = sum_iota gamma_j[iota] * (phi~_{p_r} (.) a_tt)[iota],
// the 16x16x32 bf16 MFMA with Gamma_l as the A operand (exact +-1) and the
// sign-flipped activations as B.  B is built from the column's sign bitmap
// (nibble tables: parity is linear in the index bits) and the activations
// held in LDS in the paired coordinate order, so that each B dword is one
// rotate plus one and-or: lane kq's dword i holds coordinates
// 32c + kq + 4i (low half) and 32c + kq + 4i + 16 (high half).
#pragma once

#include "device_common.hpp"

namespace dpb {

constexpr int kScoreBatch = 8;  // A fragments fetched per batch

// A wave's activations in LDS.
struct ActTile {
    const uint32_t* pairs;  // bf16: [TPW][dp/2] |a| as bf16 pairs (paired order)
    const uint32_t* signw;  // bf16: [TPW][nchunk] sign bits, natural order (bit b = coordinate 32c + b)
    const float* f;         // fp32: [TPW][dp]
};

// Sign bitmaps of the 16 columns of block nb into cw[16][cws]; for bf16
// activations the activation signs are folded in.  Column r is parent slot
// q = r mod 2^csh of token tt = r / 2^csh, with parent parents[tt * pstride + q]
// when q < nparents and tt < ntok.  Lane
// (col, w0) builds words w0, w0 + 4, ... of column col: one nibble-table row
// per 4-bit group of the parent index (parity is linear in the index bits).
template <bool ACT_BF16>
__device__ void column_bitmaps(const DevPlan& P, int lane, int ntok, int csh, int nb, const int32_t* parents,
                               int pstride, int nparents, const ActTile& A, const uint32_t* nt, uint32_t* cw)
{
    const int nchunk = P.nchunk;
    const int col = lane & 15, r = nb * 16 + col, tt = r >> csh, q = r & ((1 << csh) - 1);
    int32_t p = -1;
    if (r < (P.wave_tokens << csh) && tt < ntok && q < nparents) p = parents[tt * pstride + q];
    // nibble table layout [g][w][16]: word w of group g for nibble value v at (g * nchunk + w) * 16 + v
    const uint32_t* rows[8];
#pragma unroll
    for (int g = 0; g < 8; ++g) rows[g] = nt + g * nchunk * 16 + ((p >> (4 * g)) & 15);
    const uint32_t* sw = A.signw + (p >= 0 ? tt : 0) * nchunk;
    uint32_t* dst = cw + col * P.cws;
    for (int w = lane >> 4; w < nchunk; w += 4) {
        uint32_t word = 0;
        if (p >= 0) {
#pragma unroll
            for (int g = 0; g < 8; ++g)
                if (g < P.nt_groups) word ^= rows[g][w * 16];
            if constexpr (ACT_BF16) word ^= sw[w];
        }
        dst[w] = word;
    }
}

// Unscaled scores of generator tile mb for this lane's column (lane & 15):
// acc[i] = S[16*mb + 4*(lane>>4) + i][column].  Columns without a parent
// produce scores of row trow that the callers discard.
template <bool ACT_BF16>
__device__ __forceinline__ void score_chunk(const DevPlan& P, int kq, u32x4 a, uint32_t wd, const uint32_t* prow,
                                            const float* frow, int c, f32x4& acc)
{
    const bf16x8 av = __builtin_bit_cast(bf16x8, a);
    if constexpr (ACT_BF16) {
        const uint32_t R = rotl32(wd, 15u - (uint32_t)kq);
        const u32x4 pd = *(const u32x4*)(prow + c * 16);
        u32x4 b;
        b.x = (R & 0x80008000u) | pd.x;
        b.y = (__builtin_amdgcn_alignbit(R, R, 4) & 0x80008000u) | pd.y;
        b.z = (__builtin_amdgcn_alignbit(R, R, 8) & 0x80008000u) | pd.z;
        b.w = (__builtin_amdgcn_alignbit(R, R, 12) & 0x80008000u) | pd.w;
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
    } else {
        uint32_t hi[8], mi[8], lo[8];
#pragma unroll
        for (int x = 0; x < 8; ++x) {
            const int off = kq + 4 * (x >> 1) + 16 * (x & 1);
            float v = frow[32 * c + off];
            v = __uint_as_float(__float_as_uint(v) ^ (((wd >> off) & 1u) << 31));
            split3(v, hi[x], mi[x], lo[x]);
        }
        const u32x4 bh = {hi[0] | (hi[1] << 16), hi[2] | (hi[3] << 16), hi[4] | (hi[5] << 16), hi[6] | (hi[7] << 16)};
        const u32x4 bm = {mi[0] | (mi[1] << 16), mi[2] | (mi[3] << 16), mi[4] | (mi[5] << 16), mi[6] | (mi[7] << 16)};
        const u32x4 bl = {lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16), lo[4] | (lo[5] << 16), lo[6] | (lo[7] << 16)};
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, bh), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, bm), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, bl), acc, 0, 0, 0);
    }
}

template <bool ACT_BF16>
__device__ f32x4 mfma_scores(const DevPlan& P, int lane, int l, int mb, int trow, const ActTile& A, const uint32_t* cw)
{
    const int nchunk = P.nchunk, dp = P.dp, col = lane & 15, kq = lane >> 4;
    const u32x4* Ap = (const u32x4*)P.gamma_pair + P.gamma_off[l] + (int64_t)mb * nchunk * 64 + lane;
    const uint32_t* cwp = cw + col * P.cws;
    const uint32_t* prow = A.pairs + trow * (dp / 2) + kq * 4;
    const float* frow = A.f + trow * dp;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    int c0 = 0;
    for (; c0 + kScoreBatch <= nchunk; c0 += kScoreBatch) {
        u32x4 a[kScoreBatch];
        uint32_t wd[kScoreBatch];
#pragma unroll
        for (int e = 0; e < kScoreBatch; ++e) {
            a[e] = Ap[(int64_t)(c0 + e) * 64];
            wd[e] = cwp[c0 + e];
        }
#pragma unroll
        for (int e = 0; e < kScoreBatch; ++e) score_chunk<ACT_BF16>(P, kq, a[e], wd[e], prow, frow, c0 + e, acc);
    }
    for (; c0 < nchunk; ++c0) score_chunk<ACT_BF16>(P, kq, Ap[(int64_t)c0 * 64], cwp[c0], prow, frow, c0, acc);
    return acc;
}

// Writes bf16 activations of `ntok` rows (row stride d elements) into the
// paired layout and the sign words; rows >= ntok and coordinates >= d are 0.
// Each lane reads 8 consecutive coordinates (one 16-byte load when d is a
// multiple of 8) and scatters them as half-words.
__device__ inline void load_pairs(const DevPlan& P, int lane, int ntok, int tpw, const uint16_t* src, int64_t row0,
                                  uint32_t* pairs, uint32_t* signw)
{
    const int d = P.d, dp = P.dp, nchunk = P.nchunk;
    uint16_t* ph = (uint16_t*)pairs;
    const bool vec = (d & 7) == 0;
    for (int tt = 0; tt < tpw; ++tt) {
        const bool live = tt < ntok;
        const uint16_t* row = src + (row0 + tt) * d;
        for (int o = lane * 8; o < dp; o += 512) {
            uint32_t v[4] = {0u, 0u, 0u, 0u};
            if (live && vec && o < d) {
                const u32x4 q = *(const u32x4*)(row + o);
                v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
            } else if (live) {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (o + e < d) v[e >> 1] |= (uint32_t)row[o + e] << (16 * (e & 1));
            }
            // coordinate o + e sits at paired dword kq * 4 + i of chunk c, half h
            const int c = o >> 5, base = o & 31;
            uint32_t sg = 0;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const uint32_t h16 = (v[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
                const int b = base + e, h = b >> 4, kq = b & 3, i = (b >> 2) & 3;
                ph[(tt * (dp / 2) + c * 16 + kq * 4 + i) * 2 + h] = (uint16_t)(h16 & 0x7FFFu);
                sg |= (h16 >> 15) << e;
            }
            // 8 sign bits of this lane -> bits base..base+7 of word c (4 lanes per word)
            uint32_t part = sg << base;
            part |= __shfl_xor(part, 1, 64);
            part |= __shfl_xor(part, 2, 64);
            if ((lane & 3) == 0) signw[tt * nchunk + c] = part;
        }
    }
}

// Activation at coordinate iota of row tt from the paired layout.
__device__ __forceinline__ float pair_value(const DevPlan& P, const uint32_t* pairs, const uint32_t* signw, int tt,
                                            int iota)
{
    const int c = iota >> 5, b = iota & 31;
    const uint32_t dw = pairs[tt * (P.dp / 2) + c * 16 + (b & 3) * 4 + ((b >> 2) & 3)];
    const uint32_t mag = (b >> 4) ? (dw >> 16) : (dw & 0xFFFFu);
    const uint32_t sg = (signw[tt * P.nchunk + c] >> b) & 1u;
    return bf16_bits_to_f32(mag | (sg << 15));
}

}  // namespace dpb
