// Child scoring on the matrix cores (§2.2 child-scoring equation), shared by
// the encoder (activations x) and the decode-backward (upstream gradient g).
//
// For level l, a block of 16 columns r = tt*CPT + q (token tt, parent slot q)
// with parent index p_r, and a tile of 16 generators j:
//     S[j][r] = sum_iota gamma_j[iota] * (phi~_{p_r} (.) a_tt)[iota],
// the 16x16x32 bf16 MFMA with Gamma_l as the A operand (exact +-1) and the
// sign-flipped activations as B.  B is built from the column's sign bitmap
// (nibble tables: parity is linear in the index bits) and the activations
// held in LDS in the "interleaved halves" order: dword o (0..15) of chunk c
// holds coordinate 32c + o in its low half and 32c + o + 16 in its high half,
// so that each B dword is one rotate plus one bit-select.  MFMA lane kq's K
// values 8kq + 2i + h are coordinates 32c + 4kq + i + 16h.
#pragma once

#include "device_common.hpp"

namespace dpb {

constexpr int kScoreBatch = 8;  // A fragments fetched per batch (the encoder takes 6: see its call)

// A wave's activations in LDS.
struct ActTile {
    const uint32_t* pairs;  // bf16: [TPW][prow] signed bf16 pairs, interleaved halves
    const float* f;         // fp32: [TPW][dp]
};

// Sign bitmaps of the 16 columns of block nb into cw[16][cws] (bit b of word
// w = sign at coordinate 32w + b).  Column r is parent slot q = r mod 2^csh
// of token tt = r / 2^csh, with parent parents[tt * pstride + q] when
// q < nparents and tt < ntok.  Lane (col, w0) builds words w0, w0 + 4, ... of
// column col: one nibble-table row per 4-bit group of the parent index
// (parity is linear in the index bits).
__device__ void column_bitmaps(const DevPlan& P, int lane, int ntok, int csh, int nb, const int32_t* parents,
                               int pstride, int nparents, const uint32_t* nt, uint32_t* cw)
{
    constexpr int MW = 8;  // words per lane kept in registers (nchunk <= 32)
    const int nchunk = P.nchunk, w0 = lane >> 4;
    const int col = lane & 15, r = nb * 16 + col, tt = r >> csh, q = r & ((1 << csh) - 1);
    int32_t p = -1;
    if (r < (P.wave_tokens << csh) && tt < ntok && q < nparents) p = parents[tt * pstride + q];
    const uint32_t pu = p >= 0 ? (uint32_t)p : 0u;
    uint32_t* dst = cw + col * P.cws;
    // nibble table layout [g][w][16]: word w of group g for nibble value v at (g * nchunk + w) * 16 + v
    for (int wb = 0; wb < nchunk; wb += 4 * MW) {
        uint32_t acc[MW];
        int woff[MW];   // words past nchunk read the last word (in bounds) and are not stored
#pragma unroll
        for (int m = 0; m < MW; ++m) {
            acc[m] = 0;
            woff[m] = min(wb + w0 + 4 * m, nchunk - 1) * 16;
        }
        for (int g = 0; g < P.nt_groups; ++g) {
            const uint32_t* rg = nt + g * nchunk * 16 + ((pu >> (4 * g)) & 15u);
#pragma unroll
            for (int m = 0; m < MW; ++m) acc[m] ^= rg[woff[m]];
        }
#pragma unroll
        for (int m = 0; m < MW; ++m) {
            const int w = wb + w0 + 4 * m;
            if (w < nchunk) dst[w] = p >= 0 ? acc[m] : 0u;
        }
    }
}

// Unscaled scores of generator tile mb for this lane's column (lane & 15):
// acc[i] = S[16*mb + 4*(lane>>4) + i][column].  Columns without a parent
// produce scores of row trow that the callers discard.
template <bool ACT_BF16>
__device__ __forceinline__ void score_chunk(const DevPlan& P, int kq, u32x4 a, uint32_t wd, const uint32_t* prow,
                                            const float* frow, int c, f32x4& acc)
{
    (void)P;
    const bf16x8 av = __builtin_bit_cast(bf16x8, a);
    if constexpr (ACT_BF16) {
        // dword i: coordinates 4kq + i (low half) and 4kq + i + 16 (high half)
        const uint32_t R = rotl32(wd, 15u - 4u * (uint32_t)kq);
        const u32x4 pd = *(const u32x4*)(prow + c * 16);
        u32x4 b;
        b.x = pd.x ^ (R & 0x80008000u);
        b.y = pd.y ^ (__builtin_amdgcn_alignbit(R, R, 1) & 0x80008000u);
        b.z = pd.z ^ (__builtin_amdgcn_alignbit(R, R, 2) & 0x80008000u);
        b.w = pd.w ^ (__builtin_amdgcn_alignbit(R, R, 3) & 0x80008000u);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
    } else {
        uint32_t hi[8], mi[8], lo[8];
#pragma unroll
        for (int x = 0; x < 8; ++x) {
            const int off = 4 * kq + (x >> 1) + 16 * (x & 1);
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

struct NoLateLoads {
    __device__ void operator()() const {}
};

// `late` is called once, right after the loads of the last batch are issued:
// loads it issues then overlap that batch's work without holding up the
// earlier batches (memory waits are in issue order).
template <bool ACT_BF16, int SB = kScoreBatch, typename Late = NoLateLoads>
__device__ f32x4 mfma_scores(const DevPlan& P, int lane, int l, int mb, int trow, const ActTile& A, const uint32_t* cw,
                             Late late = Late())
{
    const int nchunk = P.nchunk, dp = P.dp, col = lane & 15, kq = lane >> 4;
    const u32x4* Ap = (const u32x4*)P.gamma_pair + P.gamma_off[l] + (int64_t)mb * nchunk * 64 + lane;
    const uint32_t* cwp = cw + col * P.cws;
    const uint32_t* prow = A.pairs + trow * P.prow + kq * 4;
    const float* frow = A.f + trow * dp;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    int c0 = 0;
    for (; c0 + SB <= nchunk; c0 += SB) {
        u32x4 a[SB];
        uint32_t wd[SB];
#pragma unroll
        for (int e = 0; e < SB; ++e) {
            a[e] = Ap[(int64_t)(c0 + e) * 64];
            wd[e] = cwp[c0 + e];
        }
        if (c0 + 2 * SB > nchunk) late();
#pragma unroll
        for (int e = 0; e < SB; ++e) score_chunk<ACT_BF16>(P, kq, a[e], wd[e], prow, frow, c0 + e, acc);
    }
    if (nchunk < SB) late();
    for (; c0 < nchunk; ++c0) score_chunk<ACT_BF16>(P, kq, Ap[(int64_t)c0 * 64], cwp[c0], prow, frow, c0, acc);
    return acc;
}

// Writes bf16 activations of `ntok` rows (row stride d elements) into the
// interleaved-halves layout; rows >= ntok and coordinates >= d are 0.  Lane
// 4c + h reads coordinates 32c + 8h .. 32c + 8h + 7 (one 16-byte load when d
// is a multiple of 8); lanes h and h + 2 of a quad swap two dwords so that
// each lane writes four complete dwords with one 16-byte store.
// One 8-coordinate piece (coordinates o .. o + 7) of a bf16 row, loaded by
// lane (o / 8) mod 64, stored in the interleaved-halves layout of the row prow:
// lane h < 2 of a quad keeps coordinates 8h + 0..3 and takes 16 + 8h + 0..3
// from lane h + 2; lane h + 2 keeps 16 + 8h + 4..7 and takes 8h + 4..7 from
// lane h.  Every lane of the wave must call it (lane exchanges).
__device__ __forceinline__ void store_pair_piece(int lane, u32x4 q, int o, uint32_t* prow)
{
    const int h = lane & 3;
    const bool lowq = h < 2;
    const uint32_t s0 = lowq ? q.z : q.x, s1 = lowq ? q.w : q.y;
    const uint32_t r0 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)s0, 0x4E, 0xF, 0xF, false);
    const uint32_t r1 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)s1, 0x4E, 0xF, 0xF, false);
    const uint32_t l0 = lowq ? q.x : r0, l1 = lowq ? q.y : r1;
    const uint32_t h0 = lowq ? r0 : q.z, h1 = lowq ? r1 : q.w;
    u32x4 w;
    w.x = __builtin_amdgcn_perm(h0, l0, 0x05040100u);
    w.y = __builtin_amdgcn_perm(h0, l0, 0x07060302u);
    w.z = __builtin_amdgcn_perm(h1, l1, 0x05040100u);
    w.w = __builtin_amdgcn_perm(h1, l1, 0x07060302u);
    *(u32x4*)(prow + (o >> 5) * 16 + 8 * (h & 1) + 4 * (h >> 1)) = w;
}

__device__ inline void load_pairs(const DevPlan& P, int lane, int ntok, int tpw, const uint16_t* src, int64_t row0,
                                  uint32_t* pairs)
{
    const int d = P.d, dp = P.dp;
    const bool vec = (d & 7) == 0;
    const int h = lane & 3;
    const bool lowq = h < 2;
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
            // lane h < 2 keeps coordinates 8h + 0..3 and takes 16 + 8h + 0..3 from lane h + 2;
            // lane h + 2 keeps 16 + 8h + 4..7 and takes 8h + 4..7 from lane h
            // (here and in store_pair_piece the exchange keeps a zero old
            // operand: with the plain DPP move the backward kernels measured
            // 7-14% slower on the wide workloads, same registers)
            const uint32_t s0 = lowq ? v[2] : v[0], s1 = lowq ? v[3] : v[1];
            const uint32_t r0 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)s0, 0x4E, 0xF, 0xF, false);
            const uint32_t r1 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)s1, 0x4E, 0xF, 0xF, false);
            const uint32_t l0 = lowq ? v[0] : r0, l1 = lowq ? v[1] : r1;  // low halves (coordinates < 16)
            const uint32_t h0 = lowq ? r0 : v[2], h1 = lowq ? r1 : v[3];  // high halves
            u32x4 w;
            w.x = __builtin_amdgcn_perm(h0, l0, 0x05040100u);
            w.y = __builtin_amdgcn_perm(h0, l0, 0x07060302u);
            w.z = __builtin_amdgcn_perm(h1, l1, 0x05040100u);
            w.w = __builtin_amdgcn_perm(h1, l1, 0x07060302u);
            const int c = o >> 5;
            *(u32x4*)(pairs + tt * P.prow + c * 16 + 8 * (h & 1) + 4 * (h >> 1)) = w;
        }
    }
}

// Activation at coordinate iota of row tt from the interleaved-halves layout.
__device__ __forceinline__ float pair_value(const DevPlan& P, const uint32_t* pairs, int tt, int iota)
{
    const int c = iota >> 5, b = iota & 31;
    const uint32_t dw = pairs[tt * P.prow + c * 16 + (b & 15)];
    return bf16_bits_to_f32((b >> 4) ? (dw >> 16) : (dw & 0xFFFFu));
}

}  // namespace dpb
