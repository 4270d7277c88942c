// kernels.hip -- gfx950 kernels of the mixed paged-attention iteration.
//
//   append_kernel       scatter new K/V into the paged pool (bf16 bit copy,
//                       or e4m3 quantisation with per-(block, head) scales)
//   block_copy_kernel   whole-block copy-on-write
//   attn_kernel         one wave per (work descriptor, KV head, head chunk): up
//                       to 16 query vectors against a run of 16-token blocks,
//                       online softmax, bf16 MFMA
//   merge_kernel        log-sum-exp merge of split / segment partial results
//
// MFMA tile orientation (v_mfma_f32_16x16x32_bf16, wave64):
//   S^T[key][query] = K[key][d] * Q^T[d][query]     (keys on rows)
//   O^T[d][query]  += V^T[d][key] * P^T[key][query]
// so each lane ends up owning one query column and the softmax statistics of
// that query never leave the lane's 16-lane column group.  K blocks are stored
// [16][D] and V blocks [D][16], which makes every MFMA operand a contiguous
// load straight from the pool (16 bytes, or 8 for e4m3 V).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <stdint.h>
#include <type_traits>

#include "kernels.hpp"

namespace echo {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// P.V products: bf16 (bf16 cache) or fp16 (e4m3 cache) operands, fp32 accumulate
__device__ __forceinline__ f32x4_t mfma_pv(bf16x8_t a, bf16x8_t b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mfma_pv(f16x8_t a, f16x8_t b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// ------------------------------------------------------------------- codecs

// OCP e4m3fn -> bf16, exact (every e4m3 value is a bf16 value): gfx950's
// v_cvt_scalef32_pk_bf16_fp8 with scale 1 widens two codes per instruction
// (checked on all 256 codes, NaN and signed zero included).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ bf16x8_t e4m3x8_to_bf16x8(u32x2_t w) {
    const bf16x2_t a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[0], 1.0f, false);
    const bf16x2_t b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[0], 1.0f, true);
    const bf16x2_t c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[1], 1.0f, false);
    const bf16x2_t d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[1], 1.0f, true);
    return (bf16x8_t){a[0], a[1], b[0], b[1], c[0], c[1], d[0], d[1]};
}

// fp32 -> OCP e4m3fn, round to nearest even, saturating to +-448, NaN to
// 0x7F; without branches, so that the lanes of a wave do not diverge over
// the value ranges.  Normal range (|y| >= 2^-6): round the bit pattern to 3
// mantissa bits (a carry moves into the exponent), then rebias the exponent
// (127 -> 7: minus 120 << 3); below it, steps of 2^-9 (|y| * 512 is exact).
__device__ __forceinline__ uint32_t f32_to_e4m3(float y) {
    const uint32_t u = __float_as_uint(y);
    const uint32_t sign = (u >> 24) & 0x80u;
    const uint32_t a = u & 0x7FFFFFFFu;
    const uint32_t a_sat = a < 0x43E00000u ? a : 0x43E00000u;            // |y| >= 448, inf -> 448
    const uint32_t cn = ((a_sat + 0x7FFFFu + ((a_sat >> 20) & 1u)) >> 20) - 960u;
    const uint32_t cs = (uint32_t)__builtin_rintf(__uint_as_float(a) * 512.0f);
    const uint32_t code = sign | (a < 0x3C800000u ? cs : (cn < 0x7Eu ? cn : 0x7Eu));
    return a > 0x7F800000u ? 0x7Fu : code;
}

// The quotient RN(x / s) that the quantisation takes, for a divisor s shared
// by a whole (block, head) tile: from r = RN(1 / s), q0 = RN(x r), the exact
// residual e = x - q0 s (one FMA) and the corrected q1 = RN(q0 + e r)
// (Markstein's final correction step).  For s in [2^-100, 2^100] this gives
// the same e4m3 code as the correctly rounded quotient for every finite bf16
// x (checked exhaustively on the CPU over x and every scale fp32(b / 448), b
// a positive bf16); quotients past 512 saturate either way and keep q0, and
// the sign is q0's (a zero x keeps its sign).  Other scales divide.
struct Recip {
    float s, r;
    bool fast;
};
__device__ __forceinline__ Recip recip_of(float s) {
    return {s, 1.0f / s, s >= 0x1p-100f && s <= 0x1p100f};
}
__device__ __forceinline__ float quotient(float x, const Recip &d) {
    if (!d.fast) return x / d.s;
    const float q0 = x * d.r;
    const float e = __builtin_fmaf(-q0, d.s, x);
    const float q1 = __builtin_fmaf(e, d.r, q0);
    return __builtin_copysignf(__builtin_fabsf(q0) < 512.0f ? q1 : q0, q0);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// v_max_f32 as such: fmaxf adds a canonicalising max of each operand the
// compiler cannot prove canonical (lane-swap results are not), two extra VALU
// ops per call.  Used on attention scores, which are finite or -inf.
__device__ __forceinline__ float vmax(float a, float b) {
    float r;
    asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
// max over lanes l, l^16, l^32, l^48 with VALU lane swaps (no LDS traffic):
// each swap returns the lane's own value and its partner's, in some order.
__device__ __forceinline__ float wave_max_xor16_32(float x) {
    typedef uint32_t u2 __attribute__((ext_vector_type(2)));
    const u2 a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = vmax(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const u2 b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return vmax(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// ------------------------------------------------------------------- append

// One work unit = (row, written block, KV head).  Units are enumerated
// without host help: every workgroup scans the rows' written-block counts
// into LDS (windows of kAppWin rows), then each wave takes every n-th unit of
// the window and finds its row by binary search over the prefix.
constexpr int kAppWin = 2048;

// exclusive prefix of cnt[0..n) in place (n <= kAppWin); returns the total
__device__ __forceinline__ int block_scan_window(int32_t *cnt, int n, int32_t *wsum) {
    constexpr int PER = kAppWin / 256;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    int loc = 0;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
        const int i = t * PER + k;
        loc += i < n ? cnt[i] : 0;
    }
    int inc = loc;  // inclusive scan over the wave
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(inc, off);
        if (lane >= off) inc += y;
    }
    if (lane == 63) wsum[wave] = inc;
    __syncthreads();
    int before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        before += w < wave ? wsum[w] : 0;
        total += wsum[w];
    }
    int run = before + inc - loc;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
        const int i = t * PER + k;
        if (i < n) {
            const int c = cnt[i];
            cnt[i] = run;
            run += c;
        }
    }
    __syncthreads();
    return total;
}

// Lane (m, part) = (lane / 4, lane % 4) carries slot m's token: the quarter
// `part` of its K and V rows (D / 4 values).  Slot m holds position 16j + m
// and is written when m_lo <= m < m_hi.  K rows go straight to the pool;
// V rows are transposed through the wave's LDS tile to [d][16 slots] and
// written as whole 16-slot rows when the block is full, else slot by slot.
// e4m3: a block that is not written whole (a decode row's slot) quantises
// only its written slots, each slot's K and V rows spread over all 64 lanes.
template <int D, bool FP8>
__device__ __forceinline__ void append_unit(const AppendArgs &a, int r, int j, int h, int lane,
                                            uint16_t *tr, int t0, int p0, int L) {
    if (j >= a.max_blocks_per_row) return;
    const int blk = a.block_tables[(int64_t)r * a.max_blocks_per_row + j];
    if (blk < 0 || blk >= a.num_blocks) return;
    const int sb = 16 * j;
    const int m_lo = max(p0, sb) - sb, m_hi = min(L, sb + 16) - sb;   // written slots
    const bool full = m_lo == 0 && m_hi == 16;
    const int m = lane >> 2, part = lane & 3;
    const bool mine = m >= m_lo && m < m_hi;
    constexpr int QW = D / 32;        // 16-byte words per quarter row
    const int64_t tok_stride = (int64_t)a.num_kv_heads * D;
    const int64_t row_src = (int64_t)(t0 + sb - p0 + m) * tok_stride + (int64_t)h * D + part * (D / 4);
    const int64_t tile = ((int64_t)blk * a.num_kv_heads + h) * 16 * D;

    u32x4_t kw[QW], vw[QW];
#pragma unroll
    for (int w = 0; w < QW; ++w) {
        kw[w] = vw[w] = (u32x4_t){0u, 0u, 0u, 0u};
        if (mine) {
            kw[w] = *(const u32x4_t *)(a.k_new + row_src + 8 * w);
            vw[w] = *(const u32x4_t *)(a.v_new + row_src + 8 * w);
        }
    }
    // stage V as [slot][D] bf16 in this wave's LDS tile, read back by d
    if (mine) {
#pragma unroll
        for (int w = 0; w < QW; ++w) *(u32x4_t *)(tr + m * D + part * (D / 4) + 8 * w) = vw[w];
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    constexpr int DPL = D / 64;       // d rows of V^T per lane
    uint32_t col[16];                 // slot s of this lane's d rows (DPL bf16 each)
#pragma unroll
    for (int s2 = 0; s2 < 16; ++s2) {
        if constexpr (DPL == 2) col[s2] = *(const uint32_t *)(tr + s2 * D + 2 * lane);
        else col[s2] = tr[s2 * D + lane];
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");

    if constexpr (!FP8) {
        uint16_t *kdst = (uint16_t *)a.k + tile;
        uint16_t *vdst = (uint16_t *)a.v + tile;
        if (mine) {
#pragma unroll
            for (int w = 0; w < QW; ++w) *(u32x4_t *)(kdst + m * D + part * (D / 4) + 8 * w) = kw[w];
        }
#pragma unroll
        for (int e = 0; e < DPL; ++e) {
            uint16_t *row = vdst + (lane * DPL + e) * 16;
            if (full) {
                uint32_t pk[8];
#pragma unroll
                for (int m2 = 0; m2 < 8; ++m2)
                    pk[m2] = ((col[2 * m2] >> (16 * e)) & 0xFFFFu) |
                             (((col[2 * m2 + 1] >> (16 * e)) & 0xFFFFu) << 16);
                *(u32x4_t *)row = (u32x4_t){pk[0], pk[1], pk[2], pk[3]};
                *(u32x4_t *)(row + 8) = (u32x4_t){pk[4], pk[5], pk[6], pk[7]};
            } else {
                // the written slots only: 2-byte stores at fixed offsets from the row
#pragma unroll
                for (int s2 = 0; s2 < 16; ++s2)
                    if (s2 >= m_lo && s2 < m_hi) row[s2] = (uint16_t)(col[s2] >> (16 * e));
            }
        }
    } else {
        uint8_t *kdst = (uint8_t *)a.k + tile;
        uint8_t *vdst = (uint8_t *)a.v + tile;
        const int64_t si = (int64_t)blk * a.num_kv_heads + h;
        float sk, sv;
        if (m_lo == 0) {  // slot 0 written by this call: fresh scales
            float ak = 0.f, av = 0.f;
#pragma unroll
            for (int w = 0; w < QW; ++w)
#pragma unroll
                for (int x = 0; x < 4; ++x) {
                    ak = fmaxf(ak, fmaxf(fabsf(bf16_bits_to_f32(kw[w][x] & 0xFFFFu)),
                                         fabsf(bf16_bits_to_f32(kw[w][x] >> 16))));
                    av = fmaxf(av, fmaxf(fabsf(bf16_bits_to_f32(vw[w][x] & 0xFFFFu)),
                                         fabsf(bf16_bits_to_f32(vw[w][x] >> 16))));
                }
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) {
                ak = fmaxf(ak, __shfl_xor(ak, off));
                av = fmaxf(av, __shfl_xor(av, off));
            }
            sk = ak == 0.f ? 1.f : ak / 448.0f;
            sv = av == 0.f ? 1.f : av / 448.0f;
            if (lane == 0) {
                a.k_scale[si] = sk;
                a.v_scale[si] = sv;
            }
        } else {
            sk = a.k_scale[si];
            sv = a.v_scale[si];
        }
        const Recip dk = recip_of(sk), dv = recip_of(sv);
        if (!full) {
            // the written slots only, each K row spread over the whole wave
            // (DPL values per lane), as V below
#pragma unroll
            for (int s2 = 0; s2 < 16; ++s2) {
                if (s2 < m_lo || s2 >= m_hi) continue;
                const uint16_t *kp = a.k_new + (int64_t)(t0 + sb - p0 + s2) * tok_stride +
                                     (int64_t)h * D + lane * DPL;
                const uint32_t w = DPL == 2 ? *(const uint32_t *)kp : (uint32_t)*kp;
                uint32_t c = 0;
#pragma unroll
                for (int e = 0; e < DPL; ++e)
                    c |= f32_to_e4m3(quotient(bf16_bits_to_f32((w >> (16 * e)) & 0xFFFFu), dk)) << (8 * e);
                if constexpr (DPL == 2) *(uint16_t *)(kdst + s2 * D + lane * 2) = (uint16_t)c;
                else kdst[s2 * D + lane] = (uint8_t)c;
            }
        } else if (mine) {
            // 8 codes per 16-byte bf16 word
#pragma unroll
            for (int w = 0; w < QW; ++w) {
                uint32_t c[2] = {0u, 0u};
#pragma unroll
                for (int x = 0; x < 4; ++x) {
                    const uint32_t lo8 = f32_to_e4m3(quotient(bf16_bits_to_f32(kw[w][x] & 0xFFFFu), dk));
                    const uint32_t hi8 = f32_to_e4m3(quotient(bf16_bits_to_f32(kw[w][x] >> 16), dk));
                    c[x >> 1] |= (lo8 | (hi8 << 8)) << (16 * (x & 1));
                }
                *(u32x2_t *)(kdst + m * D + part * (D / 4) + 8 * w) = (u32x2_t){c[0], c[1]};
            }
        }
        auto vcode = [&](int s2, int e) -> uint32_t {
            return f32_to_e4m3(quotient(bf16_bits_to_f32((col[s2] >> (16 * e)) & 0xFFFFu), dv));
        };
#pragma unroll
        for (int e = 0; e < DPL; ++e) {
            uint8_t *row = vdst + (lane * DPL + e) * 16;
            if (full) {
                uint32_t pk[4];
#pragma unroll
                for (int m2 = 0; m2 < 4; ++m2)
                    pk[m2] = vcode(4 * m2, e) | (vcode(4 * m2 + 1, e) << 8) |
                             (vcode(4 * m2 + 2, e) << 16) | (vcode(4 * m2 + 3, e) << 24);
                *(u32x4_t *)row = (u32x4_t){pk[0], pk[1], pk[2], pk[3]};
            } else {
                // the written slots only (the same for the whole wave): a decode
                // row's unit quantises one slot, not sixteen
#pragma unroll
                for (int s2 = 0; s2 < 16; ++s2)
                    if (s2 >= m_lo && s2 < m_hi) row[s2] = (uint8_t)vcode(s2, e);
            }
        }
    }
}

template <int D, bool FP8>
__global__ __launch_bounds__(256) void append_kernel(AppendArgs a) {
    __shared__ int32_t pre[kAppWin];                  // exclusive prefix of written blocks
    __shared__ int32_t rt0[kAppWin], rp0[kAppWin], rL[kAppWin];   // first token, start, length
    __shared__ int32_t wsum[4];
    __shared__ __attribute__((aligned(16))) uint16_t vstage[4][16 * D];
    const int lane = threadIdx.x & 63;
    const int64_t gw = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int64_t nw = (int64_t)gridDim.x * 4;
    const int H = a.num_kv_heads;
    int64_t done = 0;  // units of earlier windows
    for (int r0 = 0; r0 < a.num_rows; r0 += kAppWin) {
        const int nr = min(kAppWin, a.num_rows - r0);
        for (int i = threadIdx.x; i < nr; i += 256) {
            const int r = r0 + i;
            const int q = a.q_start[r + 1] - a.q_start[r];
            const int L = a.seq_lens[r];
            const int p0 = L - q;
            const int jlast = min((L - 1) / 16, a.max_blocks_per_row - 1);
            pre[i] = (q > 0 && p0 >= 0 && jlast >= p0 / 16) ? jlast - p0 / 16 + 1 : 0;
            rt0[i] = a.q_start[r];
            rp0[i] = p0;
            rL[i] = L;
        }
        __syncthreads();
        const int nblk = block_scan_window(pre, nr, wsum);
        const int64_t units = (int64_t)nblk * H;
        // this wave's units of the window: global indices done + u = gw (mod nw)
        int64_t u = (gw - done) % nw;
        if (u < 0) u += nw;
        for (; u < units; u += nw) {
            const int bu = (int)(u / H);
            const int h = (int)(u - (int64_t)bu * H);
            int lo = 0, hi = nr - 1;  // last row i with pre[i] <= bu
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (pre[mid] <= bu) lo = mid;
                else hi = mid - 1;
            }
            const int p0 = rp0[lo];
            append_unit<D, FP8>(a, r0 + lo, p0 / 16 + (bu - pre[lo]), h, lane, vstage[threadIdx.x >> 6],
                                rt0[lo], p0, rL[lo]);
        }
        done += units;
        __syncthreads();  // pre is rewritten by the next window
    }
}

// Direct form for batches whose rows write few blocks each (decode-heavy):
// one wave per (row, k-th written block, KV head) of a padded grid, no scan,
// no LDS, so many waves stay resident.  Same results as append_kernel.
template <int D, bool FP8>
__global__ __launch_bounds__(256) void append_rows_kernel(AppendArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t unit = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (unit >= a.n_units) return;
    const int H = a.num_kv_heads;
    const int h = (int)(unit % H);
    const int64_t rest = unit / H;
    const int k = (int)(rest % a.blocks_per_row);
    const int r = (int)(rest / a.blocks_per_row);
    const int t0 = a.q_start[r];
    const int q = a.q_start[r + 1] - t0;
    const int L = a.seq_lens[r];
    const int p0 = L - q;
    if (q <= 0 || p0 < 0) return;
    const int j = p0 / 16 + k;
    if (j > (L - 1) / 16 || j >= a.max_blocks_per_row) return;
    const int blk = a.block_tables[(int64_t)r * a.max_blocks_per_row + j];
    if (blk < 0 || blk >= a.num_blocks) return;
    const int lo = max(p0, 16 * j), n = min(L, 16 * j + 16) - lo;   // tokens written
    const int64_t tok_stride = (int64_t)H * D;
    const int64_t src = (int64_t)(t0 + lo - p0) * tok_stride + (int64_t)h * D;
    const int64_t tile = ((int64_t)blk * H + h) * 16 * D;
    constexpr int LPT = D / 8, TPP = 64 / LPT;   // K: lanes of 16 bytes per row, rows per pass
    constexpr int DPL = D / 64;                  // V: d values per lane
    const int kr = lane / LPT, kc = (lane % LPT) * 8;
    if constexpr (!FP8) {
        uint16_t *kdst = (uint16_t *)a.k + tile;
        uint16_t *vdst = (uint16_t *)a.v + tile;
        for (int i = kr; i < n; i += TPP)
            *(u32x4_t *)(kdst + ((lo + i) & 15) * D + kc) =
                *(const u32x4_t *)(a.k_new + src + i * tok_stride + kc);
        for (int i = 0; i < n; ++i) {
            const uint16_t *vp = a.v_new + src + i * tok_stride + lane * DPL;
            const uint32_t w = DPL == 2 ? *(const uint32_t *)vp : (uint32_t)*vp;
            const int slot = (lo + i) & 15;
#pragma unroll
            for (int e = 0; e < DPL; ++e) vdst[(lane * DPL + e) * 16 + slot] = (uint16_t)(w >> (16 * e));
        }
    } else {
        uint8_t *kdst = (uint8_t *)a.k + tile;
        uint8_t *vdst = (uint8_t *)a.v + tile;
        const int64_t si = (int64_t)blk * H + h;
        float sk, sv;
        if (16 * j >= p0) {  // slot 0 written by this call: fresh scales
            float ak = 0.f, av = 0.f;
            for (int i = 0; i < n; ++i)
#pragma unroll
                for (int e = 0; e < DPL; ++e) {
                    const int d = lane * DPL + e;
                    ak = fmaxf(ak, fabsf(bf16_bits_to_f32(a.k_new[src + i * tok_stride + d])));
                    av = fmaxf(av, fabsf(bf16_bits_to_f32(a.v_new[src + i * tok_stride + d])));
                }
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) {
                ak = fmaxf(ak, __shfl_xor(ak, off));
                av = fmaxf(av, __shfl_xor(av, off));
            }
            sk = ak == 0.f ? 1.f : ak / 448.0f;
            sv = av == 0.f ? 1.f : av / 448.0f;
            if (lane == 0) {
                a.k_scale[si] = sk;
                a.v_scale[si] = sv;
            }
        } else {
            sk = a.k_scale[si];
            sv = a.v_scale[si];
        }
        const Recip dk = recip_of(sk), dv = recip_of(sv);
        for (int i = 0; i < n; ++i) {
            const int slot = (lo + i) & 15;
#pragma unroll
            for (int e = 0; e < DPL; ++e) {
                const int d = lane * DPL + e;
                kdst[slot * D + d] =
                    (uint8_t)f32_to_e4m3(quotient(bf16_bits_to_f32(a.k_new[src + i * tok_stride + d]), dk));
                vdst[d * 16 + slot] =
                    (uint8_t)f32_to_e4m3(quotient(bf16_bits_to_f32(a.v_new[src + i * tok_stride + d]), dv));
            }
        }
    }
}

// --------------------------------------------------------------- block copy

__global__ __launch_bounds__(256) void block_copy_kernel(BlockCopyArgs a) {
    const int64_t unit = blockIdx.x;
    const int pair = (int)(unit / a.chunks);
    const int chunk = (int)(unit % a.chunks);
    if (pair >= a.n_pairs) return;
    const int src = a.pairs[2 * pair], dst = a.pairs[2 * pair + 1];
    if (src < 0 || src >= a.num_blocks || dst < 0 || dst >= a.num_blocks) return;
    const int64_t words = a.block_bytes / 16;
    const u32x4_t *ks = (const u32x4_t *)((const uint8_t *)a.k + (int64_t)src * a.block_bytes);
    const u32x4_t *vs = (const u32x4_t *)((const uint8_t *)a.v + (int64_t)src * a.block_bytes);
    u32x4_t *kd = (u32x4_t *)((uint8_t *)a.k + (int64_t)dst * a.block_bytes);
    u32x4_t *vd = (u32x4_t *)((uint8_t *)a.v + (int64_t)dst * a.block_bytes);
    const int64_t base = (int64_t)chunk * 1024;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int64_t w = base + e * 256 + threadIdx.x;
        if (w < words) {
            kd[w] = ks[w];
            vd[w] = vs[w];
        }
    }
    if (a.k_scale && chunk == 0) {
        for (int h = threadIdx.x; h < a.num_kv_heads; h += 256) {
            a.k_scale[(int64_t)dst * a.num_kv_heads + h] = a.k_scale[(int64_t)src * a.num_kv_heads + h];
            a.v_scale[(int64_t)dst * a.num_kv_heads + h] = a.v_scale[(int64_t)src * a.num_kv_heads + h];
        }
    }
}

// ---------------------------------------------------------------- attention

// Read-only metadata (work descriptors, block tables) through the constant
// address space: nothing writes it while a kernel runs, so wave-uniform reads
// are scalar loads wherever they sit in the kernel.
typedef const __attribute__((address_space(4))) int32_t const_i32;
__device__ __forceinline__ int32_t ro_load(const int32_t *p, int64_t i) {
    return ((const_i32 *)p)[i];
}

// Pool loads: streamed past the L2 (non-temporal) when no other wave reads
// the same keys, ordinary otherwise.
template <bool B>
struct Flag {
    static constexpr bool value = B;
};
template <bool NT, typename R>
__device__ __forceinline__ R pool_load(const void *p) {
    if constexpr (NT) return __builtin_nontemporal_load((const R *)p);
    else return *(const R *)p;
}

// Per-dtype pieces of the decode kernel.  A lane's K operand for the 32-wide
// contraction chunk c is 8 values of d; which 8 is free as long as Q uses the
// same assignment.  bf16 takes d = 32c + 8*g4 (one 16-byte load per chunk);
// e4m3 takes d = 64(c/2) + 16*g4 + 8(c%2), so one 16-byte load of 16 codes
// feeds two chunks and every K load is 16 bytes wide for both dtypes.
template <bool FP8>
struct KV;
template <>
struct KV<false> {
    typedef uint16_t T;
    typedef u32x4_t VRaw;                   // 8 keys of one V^T row
    static constexpr int KSTEP = 32;        // elements between a lane's K loads
    static constexpr int KLANE = 8;         // elements per 16-lane group and load
    static __device__ __forceinline__ int q_off(int c, int g4) { return 32 * c + 8 * g4; }
    static __device__ __forceinline__ bf16x8_t k_chunk(const u32x4_t *kr, int c) {
        return __builtin_bit_cast(bf16x8_t, kr[c]);
    }
    static __device__ __forceinline__ bf16x8_t widen(VRaw r) { return __builtin_bit_cast(bf16x8_t, r); }
    // zero element e (0..7) where bit e of keep is clear
    static __device__ __forceinline__ VRaw mask(VRaw r, uint32_t keep) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const uint32_t m = ((keep >> (2 * w)) & 1u ? 0x0000FFFFu : 0u) |
                               ((keep >> (2 * w + 1)) & 1u ? 0xFFFF0000u : 0u);
            r[w] &= m;
        }
        return r;
    }
};
template <>
struct KV<true> {
    typedef uint8_t T;
    typedef u32x2_t VRaw;                   // 8 e4m3 keys of one V^T row
    static constexpr int KSTEP = 64;
    static constexpr int KLANE = 16;
    static __device__ __forceinline__ int q_off(int c, int g4) {
        return 64 * (c >> 1) + 16 * g4 + 8 * (c & 1);
    }
    static __device__ __forceinline__ bf16x8_t k_chunk(const u32x4_t *kr, int c) {
        const u32x4_t w = kr[c >> 1];
        return e4m3x8_to_bf16x8((c & 1) ? (u32x2_t){w[2], w[3]} : (u32x2_t){w[0], w[1]});
    }
    static __device__ __forceinline__ bf16x8_t widen(VRaw r) { return e4m3x8_to_bf16x8(r); }
    static __device__ __forceinline__ VRaw mask(VRaw r, uint32_t keep) {
#pragma unroll
        for (int w = 0; w < 2; ++w) {
            uint32_t m = 0;
#pragma unroll
            for (int b = 0; b < 4; ++b) m |= ((keep >> (4 * w + b)) & 1u) ? (0xFFu << (8 * b)) : 0u;
            r[w] &= m;
        }
        return r;
    }
};

// Logical workgroup of physical workgroup P.  Workgroups are dispatched to
// the 8 XCDs round-robin (P mod 8); this order gives each XCD runs of
// 2^run_log2 consecutive logical workgroups, so the sibling waves of a shared
// segment (consecutive descriptors) read its blocks through one L2.  Runs are
// dealt to the XCDs in rounds of 8, in reverse order every other round: the
// work list is sorted heavy-first, so a plain round-robin deal would give XCD 0
// the heaviest run of every round (5-10% more work than XCD 7 on the batches
// measured) and the kernel would end when XCD 0 does.  Runs are 16 workgroups,
// shorter on small grids so that every XCD gets several.  The grid is a
// multiple of 8 runs, so the map is a permutation of the grid.
__device__ __forceinline__ int dec_logical(int P, int run_log2) {
    const int q = P >> 3, x = P & 7;
    const int round = q >> run_log2;
    const int xr = (round & 1) ? 7 - x : x;
    return ((round * 8 + xr) << run_log2) + (q & ((1 << run_log2) - 1));
}

// One decode workgroup of four waves: P is its physical workgroup index in
// the decode order (dec_logical), tid its thread index in [0, 256).
// Decode waves are bound by the CU's texture address units, and the SIMD
// issues the oldest ready wave first, so of three resident waves the oldest
// streams about twice as fast as the youngest.  Each wave therefore sets its
// issue priority from the 32-key steps it has left (longest remaining work
// first), which evens out the end times the planner assumes equal.
#ifndef ECHO_DEC_PRIO
#define ECHO_DEC_PRIO 24, 12, 6
#endif
constexpr int kDecPrio[3] = {ECHO_DEC_PRIO};   // steps left for priority 3, 2, 1

template <int D, bool FP8>
__device__ __forceinline__ void decode_body(const AttnArgs &a, int P, int tid) {
    typedef KV<FP8> kv;
    typedef typename kv::T KT;
    typedef typename kv::VRaw VRaw;
    constexpr int NC = D / 32;            // 32-wide d chunks of the QK contraction
    constexpr int NT = D / 16;            // 16-row d tiles of O^T
    constexpr int NK = D / kv::KSTEP;     // 16-byte K loads per key row and lane

    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t idx = (int64_t)dec_logical(P, a.run_log2) * 4 + wave;
    if (idx >= a.n_waves) return;
    if (a.counts && idx >= (int64_t)ro_load(a.counts, kHdrDesc) * a.waves_per_desc) return;
    const int di = (int)(idx / a.waves_per_desc);
    const int rem = (int)(idx - (int64_t)di * a.waves_per_desc);
    const int kvh = rem / a.head_chunks;
    const int hc = rem - kvh * a.head_chunks;
    const int32_t *ip = (const int32_t *)(a.desc + di);
    const int tok_off = __builtin_amdgcn_readfirstlane(ro_load(ip, 0));
    const int shape = __builtin_amdgcn_readfirstlane(ro_load(ip, 1));
    const int bt_row = __builtin_amdgcn_readfirstlane(ro_load(ip, 2));
    const int key_begin = __builtin_amdgcn_readfirstlane(ro_load(ip, 3));
    const int key_end = __builtin_amdgcn_readfirstlane(ro_load(ip, 4));
    const int dpart = __builtin_amdgcn_readfirstlane(ro_load(ip, 5));
    const int tok1 = __builtin_amdgcn_readfirstlane(ro_load(ip, 6));
    const int klim1 = __builtin_amdgcn_readfirstlane(ro_load(ip, 7));
    const int nt = shape & 0xFF;
    const int h0 = kvh * a.group + hc * 16;
    const int nh = min(a.heads_per_chunk, a.group - hc * 16);
    const int part = dpart < 0 ? -1 : dpart + rem * nt * a.heads_per_chunk;

    const int g4 = lane >> 4;   // 16-lane group: selects 8 of each 32 k-values
    const int c16 = lane & 15;  // MFMA row (A) / column (B, C) index
    const int qi = c16 / nh, qj = c16 - (c16 / nh) * nh;
    const bool qvalid = qi < nt;
    int tok = 0, klim = 0;
    if (qvalid) {
        if (nt == 1) {   // single-token slice: token and key limit ride in the descriptor
            tok = tok1;
            klim = klim1;
        } else {
            tok = a.tok_list[tok_off + qi];
            klim = a.klim[tok];
        }
    }
    const int head = h0 + qj;

    // Q^T as the B operand: column c16, the 8 d values kv::q_off(c, g4) ..
    bf16x8_t qf[NC];
    {
        const uint16_t *qp = a.q + ((int64_t)tok * a.num_q_heads + head) * D;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            u32x4_t w = {0u, 0u, 0u, 0u};
            if (qvalid) w = *(const u32x4_t *)(qp + kv::q_off(c, g4));
            qf[c] = __builtin_bit_cast(bf16x8_t, w);
        }
    }

    f32x4_t acc[NT];
#pragma unroll
    for (int i = 0; i < NT; ++i) acc[i] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;

    const int32_t *btr = a.block_tables + (int64_t)bt_row * a.max_blocks_per_row;
    const int64_t blk_stride = (int64_t)a.num_kv_heads * 16 * D;
    const KT *kbase = (const KT *)a.k + (int64_t)kvh * 16 * D;
    const KT *vbase = (const KT *)a.v + (int64_t)kvh * 16 * D;
    // S^T tile t, row c16 holds key 8*(c16>>2) + 4t + (c16&3) of the 32-key
    // window, so lane (g4, c16) receives keys 8*g4 .. 8*g4+7 of its column.
    const int ksel = c16 >= 8;
    const int kslot = 8 * ((c16 >> 2) & 1) + (c16 & 3);
    // V^T tile i, row c16 is d = 16i + c16; k-values are keys 8*g4 .. +8
    const int vsel = g4 >= 2;
    const int vslot = 8 * (g4 & 1);
    const float scale = a.scale_log2;

    auto sweep = [&](auto nt_flag) {
        constexpr bool NTL = decltype(nt_flag)::value;
        for (int kb = key_begin; kb < key_end; kb += 32) {
            const int left = (key_end - kb + 31) >> 5;
            if (left >= kDecPrio[0]) __builtin_amdgcn_s_setprio(3);
            else if (left >= kDecPrio[1]) __builtin_amdgcn_s_setprio(2);
            else if (left >= kDecPrio[2]) __builtin_amdgcn_s_setprio(1);
            else __builtin_amdgcn_s_setprio(0);
            const int jb = kb >> 4;
            const int b0 = ro_load(btr, jb);
            const bool has1 = kb + 16 < key_end;
            const int b1 = has1 ? ro_load(btr, jb + 1) : b0;
            const int kblk = ksel ? b1 : b0;
            const int vblk = vsel ? b1 : b0;

            u32x4_t kr[2][NK];
            VRaw vr[NT];
            const KT *kp = kbase + (int64_t)kblk * blk_stride + kslot * D + kv::KLANE * g4;
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int p = 0; p < NK; ++p)
                    kr[t][p] = pool_load<NTL, u32x4_t>(kp + 4 * t * D + kv::KSTEP * p);
            const KT *vp = vbase + (int64_t)vblk * blk_stride + c16 * 16 + vslot;
#pragma unroll
            for (int i = 0; i < NT; ++i) vr[i] = pool_load<NTL, VRaw>(vp + i * 256);
            // every K and V load of the step goes out before the products (left
            // to itself the compiler reuses K's registers for V and issues the
            // V loads only after the first K values arrive)
            __builtin_amdgcn_sched_barrier(0);

            f32x4_t s[2];
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                s[t] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int c = 0; c < NC; ++c)
                    s[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kv::k_chunk(kr[t], c), qf[c],
                                                                   s[t], 0, 0, 0);
            }

            float sk = scale, sv = 1.f;
            if constexpr (FP8) {
                sk = scale * a.k_scale[(int64_t)vblk * a.num_kv_heads + kvh];
                sv = a.v_scale[(int64_t)vblk * a.num_kv_heads + kvh];
            }
            const int key0 = kb + 8 * g4;
            float p[8];
            float mx = -INFINITY;
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int key = key0 + 4 * t + r;
                    const float v = s[t][r] * sk;
                    p[4 * t + r] = (key < key_end && key < klim) ? v : -INFINITY;
                    mx = fmaxf(mx, p[4 * t + r]);
                }
            mx = fmaxf(mx, __shfl_xor(mx, 16));
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float m_new = fmaxf(m_run, mx);
            const float m_use = m_new == -INFINITY ? 0.f : m_new;
            const float alpha = exp2f(m_run - m_use);
            float psum = 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                p[e] = exp2f(p[e] - m_use);
                psum += p[e];
            }
            l_run = l_run * alpha + psum;
            m_run = m_new;
#pragma unroll
            for (int i = 0; i < NT; ++i) acc[i] *= alpha;

            // e4m3: p times the V scale as a bf16 pair hi + lo (two MFMAs), so
            // that the scale is not rounded to bf16 along with every term
            bf16x8_t pf, pl;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                if constexpr (FP8) {
                    const float x = p[e] * sv;
                    pf[e] = (__bf16)x;
                    pl[e] = (__bf16)(x - (float)pf[e]);
                } else {
                    pf[e] = (__bf16)p[e];
                }
            }

            if (kb + 32 > key_end) {  // zero V columns past the end: 0 * NaN is NaN
                const int valid = key_end - key0;
                const uint32_t keep = valid >= 8 ? 0xFFu : (valid <= 0 ? 0u : ((1u << valid) - 1u));
#pragma unroll
                for (int i = 0; i < NT; ++i) vr[i] = kv::mask(vr[i], keep);
            }
#pragma unroll
            for (int i = 0; i < NT; ++i) {
                const bf16x8_t vf = kv::widen(vr[i]);
                acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, acc[i], 0, 0, 0);
                if constexpr (FP8) acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pl, acc[i], 0, 0, 0);
            }
        }
    };
    if (shape & kItemShared) sweep(Flag<false>{});
    else sweep(Flag<true>{});

    float l_tot = l_run + __shfl_xor(l_run, 16);
    l_tot += __shfl_xor(l_tot, 32);
    if (!qvalid) return;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    float *dst;
    if (part < 0) {
        dst = a.out + ((int64_t)tok * a.num_q_heads + head) * D;
    } else {
        dst = a.part_o + (int64_t)(part + c16) * D;
        if (g4 == 0) a.part_lse[part + c16] = l_tot > 0.f ? m_run + log2f(l_tot) : -INFINITY;
    }
#pragma unroll
    for (int i = 0; i < NT; ++i) *(f32x4_t *)(dst + 16 * i + 4 * g4) = acc[i] * inv;
}

template <int D, bool FP8>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
    decode_body<D, FP8>(a, blockIdx.x, threadIdx.x);
}

// ------------------------------------------------------------------ prefill
//
// One workgroup = 8 waves x 32 query vectors (consecutive tokens of one
// prefill chunk x the query heads of one KV head), one workgroup per CU.
// K/V tiles of 64 keys live in a 3-stage LDS ring as bf16 (e4m3 caches: V as
// fp16), shared by the eight waves; bf16 tiles are requested two tiles ahead:
//   K  [64 keys][D]            16-byte chunk q of row r stored at q ^ kswz(r)
//   V  [4 blocks][D/16][2][16][8]  per block and 16 rows d of V^T, keys 0-7
//                              of the 16 rows, then keys 8-15 (16 bytes each)
// kswz maps the key-row bits that differ between the 16 lanes of an MFMA
// operand read onto distinct chunks, so every 16-lane read of 16 bytes per
// lane touches all 64 LDS banks once; a 16-lane V operand read is 256
// contiguous bytes.  (Rows of 32 bytes with the halves swapped on bit 3 of d
// also spread 16 lanes over 64 banks, yet cost 4 bank-conflict cycles per
// read on gfx950, measured with SQ_LDS_BANK_CONFLICT; this layout costs none.)
// bf16 pools are copied global -> LDS directly (global_load_lds_dwordx4, no
// staging registers); e4m3 pools go through registers and are widened on the
// way in: K to bf16, V to fp16 after multiplication by its (block, head) scale
// (K scales multiply the logits instead).  Tiles of keys at or past the last
// token's position get their V entries zeroed (0 * NaN is NaN for unwritten
// slots).

constexpr int kPfKeys = 64;
constexpr int kPfLdsLimit = 160 * 1024;   // LDS of one gfx950 CU

// Workgroup shape: W waves (32 query vectors each) and an S-stage LDS ring.
#ifndef ECHO_PF_WAVES
#define ECHO_PF_WAVES 8
#endif
#ifndef ECHO_PF_STAGES
#define ECHO_PF_STAGES 3
#endif
constexpr int kPfWaves = ECHO_PF_WAVES;
constexpr int kPfThreads = 64 * kPfWaves;
constexpr int kPfStages = ECHO_PF_STAGES;
static_assert(32 * kPfWaves == kPrefillQueries, "prefill tile size");

template <int D>
struct PfLds {
    static constexpr int KBYTES = kPfKeys * 2 * D;   // K region of a stage
    static constexpr int VBYTES = 4 * 16 * D * 2;    // V region of a stage
    static constexpr int STAGE = KBYTES + VBYTES;    // bytes
    static constexpr int BYTES = kPfStages * STAGE + kPfStages * 4 * 4;  // + 4 bytes per block id
};

// s_waitcnt operand: vmcnt(n) with expcnt and lgkmcnt left free
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
// vmcnt(n) and lgkmcnt(0): also every LDS write of this wave has landed
constexpr int waitcnt_vm_lds(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4); }

typedef __attribute__((address_space(3))) void lds_void_t;

// One prefill descriptor di (a tile's tokens, or a piece of their keys) for
// KV head kvh; all kPfThreads threads of the workgroup take part.
template <int D, bool FP8>
__device__ __forceinline__ void prefill_piece(const PrefillArgs &a, int kvh, int di) {
    typedef KV<FP8> kv;
    typedef typename kv::T KT;
    typedef typename kv::VRaw Raw;   // 8 codes (16 or 8 bytes)
    typedef PfLds<D> LD;
    // P.V operand types.  e4m3: V times its block scale, and P, are fp16 (11
    // significant bits: the scaled values are not bf16-exact, and bf16's 8
    // bits would put errors up to 2^-9 |v| on rows with few keys)
    typedef std::conditional_t<FP8, _Float16, __bf16> PE;
    typedef std::conditional_t<FP8, f16x8_t, bf16x8_t> PT;
    // chunk guard of the lazy rescale (log2 units): probabilities stay below
    // 2^kGuard, inside fp16's range for e4m3
    constexpr float kGuard = FP8 ? 15.f : 64.f;
    constexpr int NC = D / 32, NT = D / 16;
    constexpr int CHUNKS = D / 8;              // 16-byte chunks per K row
    constexpr int NJ = D / (8 * kPfWaves);     // 1 KiB copies per wave per region per tile
    // chunk swizzle of K row r (see above): rows 32ch + 8(c16>>2) + 4t + (c16&3)
    // are read by lane c16, so the swizzle is a function of c16 alone
    auto kswz = [](int r) -> int {
        return D == 128 ? ((r & 3) | ((r >> 1) & 0xC)) : (((r >> 1) & 1) | ((r >> 2) & 6));
    };
    extern __shared__ __align__(16) uint8_t lds[];
    float *lscale = (float *)(lds + kPfStages * LD::STAGE);  // [stage][4]: K scales
    int32_t *lids = (int32_t *)(lscale + kPfStages * 4);      // the row's block ids

    const int32_t *dp = (const int32_t *)(a.pdesc + di);
    const int row = __builtin_amdgcn_readfirstlane(dp[0]);
    const int tok0 = __builtin_amdgcn_readfirstlane(dp[1]);
    const int ntok = __builtin_amdgcn_readfirstlane(dp[2]);
    const int key_end = __builtin_amdgcn_readfirstlane(dp[3]);
    const int key_begin = __builtin_amdgcn_readfirstlane(dp[4]);   // piece of the keys
    const int part = __builtin_amdgcn_readfirstlane(dp[5]);        // >= 0: partial results
    const int kfull = __builtin_amdgcn_readfirstlane(dp[6]);       // keys every token sees

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g4 = lane >> 4, c16 = lane & 15;
    const int G = a.group;
    // token t of the row sits at position t - (q_start[row + 1] - seq_lens[row])
    // and sees the keys up to and including it
    const int klim_base = __builtin_amdgcn_readfirstlane(a.seq_lens[row] - a.q_start[row + 1] + 1);

    // this lane's two query columns (N tiles nn = 0, 1)
    bf16x8_t qf[2][NC];
    int klim[2], qtok[2], qhead[2];
    bool qok[2];
#pragma unroll
    for (int nn = 0; nn < 2; ++nn) {
        const int qi = 32 * wave + 16 * nn + c16;
        const int tl = qi / G;
        qok[nn] = tl < ntok;
        qtok[nn] = tok0 + (qok[nn] ? tl : 0);
        qhead[nn] = kvh * G + (qi - tl * G);
        klim[nn] = qok[nn] ? klim_base + qtok[nn] : 0;
        const uint16_t *qp = a.q + ((int64_t)qtok[nn] * a.num_q_heads + qhead[nn]) * D + 8 * g4;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            u32x4_t w = {0u, 0u, 0u, 0u};
            if (qok[nn]) w = *(const u32x4_t *)(qp + 32 * c);
            qf[nn][c] = __builtin_bit_cast(bf16x8_t, w);
        }
    }

    f32x4_t acc[2][NT];
#pragma unroll
    for (int nn = 0; nn < 2; ++nn)
#pragma unroll
        for (int i = 0; i < NT; ++i) acc[nn][i] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
    float m_run[2] = {-INFINITY, -INFINITY};
    // derived from m_run, refreshed when it moves: the exponent offset
    // (-m_run, 0 while m_run is -inf) and the two lazy-rescale thresholds
    float m_neg[2] = {0.f, 0.f}, m_hig[2] = {-INFINITY, -INFINITY}, m_hi8[2] = {-INFINITY, -INFINITY};
    // The softmax denominator is a P.V product with V = 1 (every row of
    // lacc[nn] holds the column sum), so it sums exactly the rounded weights
    // that P.V uses and costs one MFMA per chunk instead of 16 adds per lane
    // (e4m3 V carries its block scale in the widened values, so the weights
    // are plain probabilities there too).
    f32x4_t lacc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
    PT ones;
#pragma unroll
    for (int e = 0; e < 8; ++e) ones[e] = (PE)1.0f;

    const int32_t *btr = a.block_tables + (int64_t)row * a.max_blocks_per_row;
    const int64_t blk_stride = (int64_t)a.num_kv_heads * 16 * D;
    const KT *kbase = (const KT *)a.k + (int64_t)kvh * 16 * D;
    const KT *vbase = (const KT *)a.v + (int64_t)kvh * 16 * D;
    const int ntiles = (key_end + kPfKeys - 1) / kPfKeys;   // tiles kt0 .. ntiles-1 of the row
    const int kt0 = key_begin / kPfKeys;
    const int kb0 = key_begin / 16, nblk = (key_end + 15) / 16 - kb0;   // blocks staged
    // keys every query of the workgroup sees: tiles below this need no mask

    // The row's block ids (up to the last key of the tile) are staged in LDS
    // once; tile block indices past the last block are clamped so that every
    // copy is unconditional (keys past key_end are zeroed or masked instead).
    for (int e = tid; e < nblk; e += kPfThreads) lids[e] = btr[kb0 + e];
    __syncthreads();
    auto blk_of = [&](int kt, int b) -> int { return lids[min(4 * (kt - kt0) + b, nblk - 1)]; };

    // This wave's NJ copies of a tile all fall in block `bsel` of the tile's
    // four; per lane, where each 16-byte piece comes from inside the block is
    // the same for every tile, so only the block id (read from LDS once per
    // tile, a step ahead, and made scalar) changes.
    static_assert((32 * D) % (NJ * 1024) == 0, "a wave's copies stay inside one block");
    const int bsel = wave * NJ * 1024 / (32 * D);
    int k_off[NJ], v_off[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int off = (wave * NJ + j) * 1024 + 16 * lane;   // byte offset in the K / V region
        const int r = off / (2 * D), q = ((off / 16) % CHUNKS) ^ kswz(r);
        k_off[j] = (r & 15) * D + 8 * q;
        // V: 16-byte unit u of the block's region holds keys 8h..8h+7 of row
        // d = 16(u / 32) + u % 16, h = (u / 16) % 2
        const int u = (off % (32 * D)) / 16;
        const int d = 16 * (u >> 5) + (u & 15), h = (u >> 4) & 1;
        v_off[j] = d * 16 + 8 * h;
    }
    auto tile_id = [&](int kt) -> int { return lids[min(4 * (kt - kt0) + bsel, nblk - 1)]; };

    Raw kreg[FP8 ? NJ : 1], vreg[FP8 ? NJ : 1];
    float sreg = 0.f, vscale = 1.f;
    auto issue_tile = [&](int kt, int buf, int id) {
        uint8_t *kl = lds + buf * LD::STAGE;
        uint8_t *vl = kl + LD::KBYTES;
        const int blk = __builtin_amdgcn_readfirstlane(id);
        const KT *kb = kbase + (int64_t)blk * blk_stride;
        const KT *vb = vbase + (int64_t)blk * blk_stride;
        if constexpr (!FP8) {
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                __builtin_amdgcn_global_load_lds((const void *)(kb + k_off[j]),
                                                 (lds_void_t *)(kl + (wave * NJ + j) * 1024), 16, 0, 0);
                __builtin_amdgcn_global_load_lds((const void *)(vb + v_off[j]),
                                                 (lds_void_t *)(vl + (wave * NJ + j) * 1024), 16, 0, 0);
            }
        } else {
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                kreg[j] = pool_load<false, Raw>(kb + k_off[j]);
                vreg[j] = pool_load<false, Raw>(vb + v_off[j]);
            }
            // the V scale of this wave's block goes into the widened values;
            // the K scales of the tile's four blocks scale the logits
            vscale = a.v_scale[(int64_t)blk * a.num_kv_heads + kvh];
            if (tid < 4) sreg = a.k_scale[(int64_t)blk_of(kt, tid) * a.num_kv_heads + kvh];
        }
    };
    // e4m3 only: widen the staged registers into LDS, V times its block's
    // scale as fp16
    auto store_tile = [&](int buf) {
        if constexpr (FP8) {
            uint8_t *kl = lds + buf * LD::STAGE;
            uint8_t *vl = kl + LD::KBYTES;
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                *(u32x4_t *)(kl + (wave * NJ + j) * 1024 + 16 * lane) =
                    __builtin_bit_cast(u32x4_t, kv::widen(kreg[j]));
                const bf16x8_t w = kv::widen(vreg[j]);
                PT v;
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = (PE)((float)w[e] * vscale);
                *(u32x4_t *)(vl + (wave * NJ + j) * 1024 + 16 * lane) = __builtin_bit_cast(u32x4_t, v);
            }
            if (tid < 4) lscale[buf * 4 + tid] = sreg;
        }
    };
    // zero V of keys at or past key_end in the tile of buffer `buf`
    auto zero_tail = [&](int kt, int buf) {
        uint16_t *vl = (uint16_t *)(lds + buf * LD::STAGE + LD::KBYTES);
        for (int e = tid; e < 4 * D * 2; e += kPfThreads) {  // 16-byte units of the four blocks
            const int b = e / (2 * D), u = e % (2 * D);
            const int key = kPfKeys * kt + 16 * b + 8 * ((u >> 4) & 1);
            uint16_t *dst = vl + b * 16 * D + 8 * u;
#pragma unroll
            for (int x = 0; x < 8; ++x)
                if (key + x >= key_end) dst[x] = 0;
        }
    };

    const float scale = a.scale_log2;
    const int ksel_row = 8 * (c16 >> 2) + (c16 & 3);  // + 4t + 32ch: S^T row -> key
    const int kswz_lane = kswz(ksel_row);

    // One 64-key tile in LDS buffer `buf`, as a two-chunk software pipeline:
    //   QK(c0) | QK(c1) + exp(c0) | PV(c0) + exp(c1) | PV(c1)
    // so that each run of MFMAs has independent VALU work to co-issue with.
    // Probabilities are taken against a reference m_run (log2 units) fixed
    // for the tile; it moves at the end of the tile when the tile's max
    // exceeds it by more than 8 (rescaling acc and l), or, before a chunk's
    // exponentials, when a chunk's max exceeds it by more than kGuard (rare
    // guard that also covers the first tile, where m_run is still -inf).
    // Both tests take any lane whose own scores cross the threshold, which is
    // the same as the column's maximum crossing it.
    auto qk = [&](const uint8_t *kl, int ch, f32x4_t (&sc)[2][2]) {
        // scheduling hint for the MFMA runs of a region (LLVM's IGroupLP mode 1,
        // single-wave small-GEMM interleave): 2-3% faster on long prefills
        __builtin_amdgcn_iglp_opt(1);
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            sc[t][0] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
            sc[t][1] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const uint8_t *krow = kl + (32 * ch + ksel_row + 4 * t) * (2 * D);
                const bf16x8_t kf = *(const bf16x8_t *)(krow + 16 * ((4 * c + g4) ^ kswz_lane));
#pragma unroll
                for (int nn = 0; nn < 2; ++nn)
                    sc[t][nn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[nn][c], sc[t][nn], 0, 0, 0);
            }
    };
    // mask, and this lane's max over its 8 raw scores of each query column in
    // log2 units (the column's max over its 4 lanes is formed only on the rare
    // rescale path); f receives the chunk's raw score -> log2 factor, which for
    // e4m3 includes the K scale of this lane's block (positive, so the max of
    // the raw scores gives the max of the scaled ones)
    auto prep = [&](int buf, int kt, int ch, bool masked, f32x4_t (&sc)[2][2], float (&mc)[2], float &f) {
        f = scale;
        if constexpr (FP8) f = scale * lscale[buf * 4 + 2 * ch + (g4 >> 1)];
        const int key0 = kPfKeys * kt + 32 * ch + 8 * g4;
#pragma unroll
        for (int nn = 0; nn < 2; ++nn) {
            float mx = -INFINITY;
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    float v = sc[t][nn][r];
                    if (masked) v = (key0 + 4 * t + r < klim[nn]) ? v : -INFINITY;
                    sc[t][nn][r] = v;
                    mx = fmaxf(mx, v);
                }
            mc[nn] = mx * f;
        }
    };
    auto rescale = [&](const float (&mnew)[2]) {
#pragma unroll
        for (int nn = 0; nn < 2; ++nn) {
            const float alpha = m_run[nn] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run[nn] - mnew[nn]);
            lacc[nn] *= alpha;
#pragma unroll
            for (int i = 0; i < NT; ++i) acc[nn][i] *= alpha;
            m_run[nn] = mnew[nn];
            m_neg[nn] = mnew[nn] == -INFINITY ? 0.f : -mnew[nn];
            m_hig[nn] = mnew[nn] + kGuard;
            m_hi8[nn] = mnew[nn] + 8.f;
        }
    };
    // exponentials of one chunk against m_run, packed to bf16 (fp16 for e4m3)
    auto expo = [&](const f32x4_t (&sc)[2][2], PT (&pf)[2], float f) {
#pragma unroll
        for (int nn = 0; nn < 2; ++nn) {
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float pe = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[t][nn][r], f, m_neg[nn]));
                    pf[nn][4 * t + r] = (PE)pe;
                }
        }
    };
    auto pv = [&](const uint8_t *vl, int ch, const PT (&pf)[2]) {
        __builtin_amdgcn_iglp_opt(1);   // as in qk
        const uint8_t *vrow = vl + (2 * ch + (g4 >> 1)) * (32 * D) + (g4 & 1) * 256 + c16 * 16;
#pragma unroll
        for (int i = 0; i < NT; ++i) {
            const PT vf = *(const PT *)(vrow + i * 16 * 32);
#pragma unroll
            for (int nn = 0; nn < 2; ++nn) acc[nn][i] = mfma_pv(vf, pf[nn], acc[nn][i]);
        }
#pragma unroll
        for (int nn = 0; nn < 2; ++nn)
            lacc[nn] = mfma_pv(ones, pf[nn], lacc[nn]);
    };
    auto tile = [&](int buf, int kt, bool masked) {
        const uint8_t *kl = lds + buf * LD::STAGE;
        const uint8_t *vl = kl + LD::KBYTES;
        f32x4_t s0[2][2], s1[2][2];
        float m0[2], m1[2], f0, f1;
        PT p0[2], p1[2];
        qk(kl, 0, s0);
        prep(buf, kt, 0, masked, s0, m0, f0);
        if (__any(m0[0] > m_hig[0] || m0[1] > m_hig[1])) {
            const float mn[2] = {fmaxf(m_run[0], wave_max_xor16_32(m0[0])),
                                 fmaxf(m_run[1], wave_max_xor16_32(m0[1]))};
            rescale(mn);
        }
        qk(kl, 1, s1);          // MFMA ...
        expo(s0, p0, f0);       // ... with the exponentials of chunk 0
        prep(buf, kt, 1, masked, s1, m1, f1);
        if (__any(m1[0] > m_hig[0] || m1[1] > m_hig[1])) {
            // chunk 0's probabilities, not yet added, move with the reference
            const float mn[2] = {fmaxf(m_run[0], wave_max_xor16_32(m1[0])),
                                 fmaxf(m_run[1], wave_max_xor16_32(m1[1]))};
#pragma unroll
            for (int nn = 0; nn < 2; ++nn) {
                const float alpha =
                    m_run[nn] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run[nn] - mn[nn]);
#pragma unroll
                for (int e = 0; e < 8; ++e) p0[nn][e] = (PE)((float)p0[nn][e] * alpha);
            }
            rescale(mn);
        }
        pv(vl, 0, p0);          // MFMA ...
        expo(s1, p1, f1);       // ... with the exponentials of chunk 1
        pv(vl, 1, p1);
        const float mt[2] = {vmax(m0[0], m1[0]), vmax(m0[1], m1[1])};
        if (__any(mt[0] > m_hi8[0] || mt[1] > m_hi8[1])) {
            const float mc[2] = {wave_max_xor16_32(mt[0]), wave_max_xor16_32(mt[1])};
            const float mn[2] = {mc[0] > m_hi8[0] ? mc[0] : m_run[0],
                                 mc[1] > m_hi8[1] ? mc[1] : m_run[1]};
            rescale(mn);
        }
    };

    // Pipeline.  bf16: iteration kt loads the block ids of tile kt+3, starts
    // the copies of tile kt+2, computes tile kt, then waits until its own
    // copies of tile kt+1 have landed (the newer ones stay in flight) and
    // meets the other waves at the barrier.  e4m3: tile kt+1 is staged in
    // registers during tile kt and widened into LDS before the barrier.
    constexpr int LA = (FP8 || kPfStages == 2) ? 1 : 2;  // tiles in flight ahead
    const int tail_tile = (kPfKeys * ntiles > key_end) ? ntiles - 1 : -1;
    // LDS buffer of tile kt: (kt - kt0) % kPfStages
    issue_tile(kt0, 0, tile_id(kt0));
    store_tile(0);
    if (LA == 2 && ntiles > kt0 + 1) issue_tile(kt0 + 1, 1, tile_id(kt0 + 1));
    int id_ahead = tile_id(kt0 + LA);   // block id of the next tile to issue
    // (e4m3 tiles reach LDS through ds_write, which the barrier does not wait
    // for: this wave's writes must have landed before others read them)
    if (LA == 2 && ntiles > kt0 + 1) __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * NJ));
    else __builtin_amdgcn_s_waitcnt(FP8 ? waitcnt_vm_lds(0) : waitcnt_vm(0));
    __builtin_amdgcn_s_barrier();
    if (tail_tile == kt0) {
        zero_tail(kt0, 0);
        __syncthreads();
    }

    auto step = [&](int kt, bool masked) {
        const int buf = (kt - kt0) % kPfStages;
        bool ahead = false;   // copies of tile kt+2 issued after those of kt+1
        if (kt + LA < ntiles) {
            issue_tile(kt + LA, (kt + LA - kt0) % kPfStages, id_ahead);
            ahead = LA == 2;
        }
        id_ahead = tile_id(kt + LA + 1);
        tile(buf, kt, masked);
        if (kt + 1 < ntiles) {
            if constexpr (LA == 1) store_tile((kt + 1 - kt0) % kPfStages);
            if (ahead) __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * NJ));
            else __builtin_amdgcn_s_waitcnt(FP8 ? waitcnt_vm_lds(0) : waitcnt_vm(0));
            __builtin_amdgcn_s_barrier();
            if (kt + 1 == tail_tile) {
                zero_tail(kt + 1, (kt + 1 - kt0) % kPfStages);
                __syncthreads();
            }
        }
    };
    // tiles every query sees in full, then the diagonal tiles with the mask
    const int nfull = min(kfull / kPfKeys, ntiles);
    for (int kt = kt0; kt < nfull; ++kt) step(kt, false);
    for (int kt = max(nfull, kt0); kt < ntiles; ++kt) step(kt, true);

#pragma unroll
    for (int nn = 0; nn < 2; ++nn) {
        const float l_tot = lacc[nn][0];
        if (!qok[nn]) continue;
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        float *dst;
        if (part < 0) {
            dst = a.out + ((int64_t)qtok[nn] * a.num_q_heads + qhead[nn]) * D + 4 * g4;
        } else {
            // the slot the merge kernel reads for (token, head) of this piece:
            // part + (kvh * head_chunks + hc) * ntok * heads_per_chunk + token * nh + jh
            const int qi = 32 * wave + 16 * nn + c16, tl = qi / G, hg = qi - tl * G;
            const int hc = hg / 16, jh = hg - 16 * hc;
            const int nh = min(a.heads_per_chunk, G - 16 * hc);
            const int64_t slot = part + (int64_t)(kvh * a.head_chunks + hc) * ntok * a.heads_per_chunk +
                                 (int64_t)tl * nh + jh;
            dst = a.part_o + slot * D + 4 * g4;
            if (g4 == 0) a.part_lse[slot] = l_tot > 0.f ? m_run[nn] + log2f(l_tot) : -INFINITY;
        }
#pragma unroll
        for (int i = 0; i < NT; ++i) *(f32x4_t *)(dst + 16 * i) = acc[nn][i] * inv;
    }
}

// One prefill workgroup: P is its physical workgroup index in the prefill
// grid (8 * per_xcd workgroups).  Its descriptor may name a second one
// (a piece of another tile's keys) that the workgroup runs next.
template <int D, bool FP8>
__device__ __forceinline__ void prefill_body(const PrefillArgs &a, int P) {
    const int L = (P % 8) * a.per_xcd + P / 8;  // consecutive logical tiles share an XCD
    if (L >= a.n_logical) return;
    const int kvh = L / a.n_pdesc;
    int di = L - kvh * a.n_pdesc;
    if (a.counts && di >= ro_load(a.counts, kHdrPdesc)) return;
    for (;;) {
        prefill_piece<D, FP8>(a, kvh, di);
        const int next = __builtin_amdgcn_readfirstlane(((const int32_t *)(a.pdesc + di))[7]);
        if (next <= 0) break;
        __syncthreads();   // the next descriptor refills the LDS ring and block ids
        di = next - 1;
    }
}

template <int D, bool FP8>
__global__ __launch_bounds__(kPfThreads, 8 / kPfWaves) void prefill_kernel(PrefillArgs a) {
    prefill_body<D, FP8>(a, blockIdx.x);
}

// -------------------------------------------------------------------- merge
//
// One wave per (merged token, 4 query heads): 16 lanes per head, each lane
// owning D/16 consecutive elements of the head's output row.  A 16-lane group
// takes its entries 16 at a time (one per lane: slot and lse loaded in
// parallel), rescales its running sums to the new maximum, then adds the
// entries' partial rows, four independent loads at a time.

template <int D>
__global__ __launch_bounds__(256) void merge_kernel(MergeArgs a) {
    constexpr int PER = D / 16;   // floats per lane
    constexpr int NV = PER / 4;   // 16-byte loads per lane and partial row
    const int lane = threadIdx.x & 63;
    const int c16 = lane & 15, base = lane & 48;
    const int64_t m = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (m >= a.n_waves) return;
    const int hgroups = (a.num_q_heads + 3) / 4;
    const int row = (int)(m / hgroups);
    if (a.counts && row >= ro_load(a.counts, kHdrMergeRows)) return;
    const int h = 4 * (int)(m - (int64_t)row * hgroups) + (lane >> 4);
    const bool hok = h < a.num_q_heads;
    const int tok = a.merge_tok[row];
    const int e0 = a.merge_ptr[row], e1 = a.merge_ptr[row + 1];
    // where head h of a slice's query i lands inside a descriptor's slots
    const int kvh = h / a.group;
    const int hc = (h - kvh * a.group) / 16;
    const int jh = h - kvh * a.group - hc * 16;
    const int nh = min(a.heads_per_chunk, a.group - hc * 16);
    const int rem = kvh * a.head_chunks + hc;
    f32x4_t acc[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) acc[k] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
    float mx = -INFINITY, wsum = 0.f;
    for (int eb = e0; eb < e1; eb += 16) {
        const int e = eb + c16;
        int slot = 0;   // entries past the end (and heads past Hq) read slot 0 with weight 0
        float lse = -INFINITY;
        if (hok && e < e1) {
            const int part = a.merge_ent[2 * e], sh = a.merge_ent[2 * e + 1];
            slot = part + rem * (sh & 0x3FF) * a.heads_per_chunk + (sh >> 10) * nh + jh;
            lse = a.part_lse[slot];
        }
        float bm = lse;
#pragma unroll
        for (int off = 8; off >= 1; off >>= 1) bm = fmaxf(bm, __shfl_xor(bm, off));
        const float m_new = fmaxf(mx, bm);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = exp2f(mx - m_use);   // 0 while mx is -inf
        const float w = lse == -INFINITY ? 0.f : exp2f(lse - m_use);
        float ws = w;
#pragma unroll
        for (int off = 8; off >= 1; off >>= 1) ws += __shfl_xor(ws, off);
        wsum = wsum * alpha + ws;
#pragma unroll
        for (int k = 0; k < NV; ++k) acc[k] *= alpha;
        mx = m_new;
        const int n = min(16, e1 - eb);
        auto load = [&](int i, f32x4_t (&v)[NV], float &wi) {
            const int si = __shfl(slot, base + i);
            wi = __shfl(w, base + i);
            const f32x4_t *po = (const f32x4_t *)(a.part_o + (int64_t)si * D + c16 * PER);
#pragma unroll
            for (int k = 0; k < NV; ++k) v[k] = po[k];
        };
        int i = 0;
        for (; i + 4 <= n; i += 4) {
            f32x4_t v[4][NV];
            float wi[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) load(i + j, v[j], wi[j]);
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int k = 0; k < NV; ++k) acc[k] += wi[j] * v[j][k];
        }
        for (; i < n; ++i) {
            f32x4_t v[NV];
            float wi;
            load(i, v, wi);
#pragma unroll
            for (int k = 0; k < NV; ++k) acc[k] += wi * v[k];
        }
    }
    if (!hok) return;
    const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
    f32x4_t *o = (f32x4_t *)(a.out + ((int64_t)tok * a.num_q_heads + h) * D + c16 * PER);
#pragma unroll
    for (int k = 0; k < NV; ++k) o[k] = acc[k] * inv;
}

// ------------------------------------------------------- device-built plan
//
// For batches given without host mirrors: the plan is built on the GPU from
// the row metadata, with no prefix grouping.  Two kernels:
//   dev_rows_kernel  one workgroup per row: checks the row's metadata and
//                    block ids and records how many decode pieces or
//                    prefill tiles it needs (-1: skipped)
//   dev_plan_kernel  one workgroup: scans those counts and writes the
//                    descriptors, merge lists and the header
// Rows whose metadata is inconsistent (or that would not fit a region, which
// only inconsistent q_start can cause) get no work and are counted in the
// header, so every kernel after them stays inside its buffers.

__global__ __launch_bounds__(256) void dev_rows_kernel(DevPlanArgs a) {
    const int r = blockIdx.x;
    const int t0 = a.q_start[r], t1 = a.q_start[r + 1];
    const int q = t1 - t0, L = a.seq_lens[r], kind = a.row_kind[r];
    bool ok = q >= 1 && L >= q && L <= a.max_seq_len && t0 >= 0 && t1 <= a.num_tokens &&
              (kind == 0 ? q == 1 : kind == 1) && (kind == 0 || L <= a.prefill_max_keys);
    const int nb = ok ? (L + 15) / 16 : 0;
    const int32_t *bt = a.block_tables + (int64_t)r * a.max_blocks_per_row;
    int bad = 0;
    for (int j = threadIdx.x; j < nb; j += 256) {
        const int id = bt[j];
        bad |= (id < 0 || id >= a.num_blocks);
    }
    bad = __syncthreads_or(bad);
    if (threadIdx.x == 0) {
        int n = -1;
        if (ok && !bad)
            n = kind == 0 ? (L + a.split_keys - 1) / a.split_keys : (q + a.tile_tokens - 1) / a.tile_tokens;
        a.row_info[r] = n;
    }
}

// exclusive scan over the 1024 threads of one workgroup of NV values per
// thread; returns the totals in tot[]
template <int NV>
__device__ __forceinline__ void scan1024(int64_t (&v)[NV], int64_t (&tot)[NV], int64_t (*wsum)[NV]) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int64_t inc[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) inc[k] = v[k];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1)
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int64_t y = __shfl_up(inc[k], off);
            if (lane >= off) inc[k] += y;
        }
    if (lane == 63)
#pragma unroll
        for (int k = 0; k < NV; ++k) wsum[wave][k] = inc[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        int64_t before = 0, all = 0;
        for (int w = 0; w < 16; ++w) {
            before += w < wave ? wsum[w][k] : 0;
            all += wsum[w][k];
        }
        v[k] = before + inc[k] - v[k];
        tot[k] = all;
    }
    __syncthreads();   // wsum is reused by the next call
}

__global__ __launch_bounds__(1024) void dev_plan_kernel(DevPlanArgs a) {
    __shared__ int64_t wsum[16][5];
    __shared__ unsigned long long used[5];   // end of the written part of each region
    __shared__ int bad_rows;
    if (threadIdx.x < 5) used[threadIdx.x] = 0;
    if (threadIdx.x == 0) bad_rows = 0;
    __syncthreads();
    const int64_t cap[5] = {a.cap_desc, a.cap_pdesc, a.cap_merge_rows, a.cap_ent, a.cap_slots};
    int64_t carry[5] = {0, 0, 0, 0, 0};
    for (int base = 0; base < a.num_rows; base += 1024) {
        const int r = base + (int)threadIdx.x;
        int info = -2, kind = 0;
        if (r < a.num_rows) {
            info = a.row_info[r];
            kind = a.row_kind[r];
        }
        const int dec = (info > 0 && kind == 0) ? info : 0;
        const int pf = (info > 0 && kind == 1) ? info : 0;
        // counts: decode pieces, prefill tiles, merged tokens, merge entries, slots
        int64_t v[5] = {dec, pf, dec > 1 ? 1 : 0, dec > 1 ? dec : 0,
                        dec > 1 ? (int64_t)dec * a.slots_per_desc : 0};
        const int64_t n[5] = {v[0], v[1], v[2], v[3], v[4]};
        int64_t tot[5];
        scan1024<5>(v, tot, wsum);
        int64_t off[5];
        bool fits = true;
#pragma unroll
        for (int k = 0; k < 5; ++k) {
            off[k] = carry[k] + v[k];
            fits = fits && off[k] + n[k] <= cap[k];
            carry[k] += tot[k];
        }
        if (r < a.num_rows && (info == -1 || !fits)) atomicAdd(&bad_rows, 1);
        if (r < a.num_rows && fits && (dec > 0 || pf > 0)) {
#pragma unroll
            for (int k = 0; k < 5; ++k)
                if (n[k] > 0) atomicMax(&used[k], (unsigned long long)(off[k] + n[k]));
            const int t0 = a.q_start[r];
            const int L = a.seq_lens[r];
            for (int p = 0; p < dec; ++p) {
                WorkDesc d;
                d.tok_off = 0;
                d.shape = 1;
                d.bt_row = r;
                d.key_begin = p * a.split_keys;
                d.key_end = min((p + 1) * a.split_keys, L);
                d.part = dec > 1 ? (int32_t)(off[4] + (int64_t)p * a.slots_per_desc) : -1;
                d.tok1 = t0;
                d.klim1 = L;
                a.desc[off[0] + p] = d;
            }
            if (dec > 1) {
                a.merge_tok[off[2]] = t0;
                a.merge_ptr[off[2]] = (int32_t)off[3];
                for (int p = 0; p < dec; ++p) {
                    a.merge_ent[2 * (off[3] + p)] = (int32_t)(off[4] + (int64_t)p * a.slots_per_desc);
                    a.merge_ent[2 * (off[3] + p) + 1] = 1;   // a one-token slice, query 0
                }
            }
            const int q = a.q_start[r + 1] - t0, c = L - q;
            for (int k = 0; k < pf; ++k) {   // the tile with the most keys first
                const int kk = pf - 1 - k;
                PrefillDesc d;
                d.row = r;
                d.tok0 = t0 + kk * a.tile_tokens;
                d.ntok = min(a.tile_tokens, q - kk * a.tile_tokens);
                d.key_end = c + kk * a.tile_tokens + d.ntok;
                d.key_begin = 0;
                d.part = -1;
                d.kfull = d.key_end - d.ntok + 1;
                d.next = 0;
                a.pdesc[off[1] + k] = d;
            }
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        a.hdr[kHdrDesc] = (int32_t)used[0];
        a.hdr[kHdrPdesc] = (int32_t)used[1];
        a.hdr[kHdrMergeRows] = (int32_t)used[2];
        a.hdr[kHdrSlots] = (int32_t)used[4];
        a.hdr[kHdrBadRows] = bad_rows;
        a.merge_ptr[used[2]] = (int32_t)used[3];
    }
}

hipError_t launch_dev_plan(const DevPlanArgs &a, hipStream_t s) {
    if (a.num_rows <= 0) return hipSuccess;
    hipLaunchKernelGGL(dev_rows_kernel, dim3((unsigned)a.num_rows), dim3(256), 0, s, a);
    hipLaunchKernelGGL(dev_plan_kernel, dim3(1), dim3(1024), 0, s, a);
    return hipGetLastError();
}

// ----------------------------------------------------------- static scratch
//
// Device memory of echo_attn_mixed_static: the plan and partial results of
// a device-planned call live here instead of in a caller's workspace.  Each
// GPU the library runs on holds its own copy for the life of the process.
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

// Address of this device's copy of `scratch`, looked up once per device
// with that device current (in host code the array's name is not a device
// address).
hipError_t scratch_region(void **ptr) {
    static std::atomic<void *> addr[64];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    void *p = addr[dev].load(std::memory_order_acquire);
    if (!p) {
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        addr[dev].store(p, std::memory_order_release);
    }
    *ptr = p;
    return hipSuccess;
}

// ------------------------------------------------------------- plan upload
//
// Copies the packed plan from pinned, coherent host memory into the
// workspace.  A kernel on the stream avoids the copy engine's hand-off with
// the kernels around it; each thread moves 16 bytes per step.
__global__ __launch_bounds__(256) void plan_upload_kernel(const uint32_t *__restrict__ src,
                                                          uint32_t *__restrict__ dst, int64_t words) {
    const int64_t n16 = words / 4;
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += stride)
        ((u32x4_t *)dst)[i] = ((const u32x4_t *)src)[i];
    const int64_t t = 4 * n16 + (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (blockIdx.x == 0 && t < words) dst[t] = src[t];
}

// ------------------------------------------------------------------ launchers

hipError_t launch_append(const AppendArgs &a, int head_dim, bool fp8, hipStream_t s) {
    if (a.n_units == 0) return hipSuccess;
    const dim3 block(256);
    if (a.blocks_per_row > 0) {   // direct form: one wave per padded (row, block, head)
        const int64_t units = (int64_t)a.num_rows * a.blocks_per_row * a.num_kv_heads;
        AppendArgs d = a;
        d.n_units = units;
        const dim3 grid((unsigned)((units + 3) / 4));
        if (head_dim == 64 && !fp8) hipLaunchKernelGGL((append_rows_kernel<64, false>), grid, block, 0, s, d);
        else if (head_dim == 64) hipLaunchKernelGGL((append_rows_kernel<64, true>), grid, block, 0, s, d);
        else if (!fp8) hipLaunchKernelGGL((append_rows_kernel<128, false>), grid, block, 0, s, d);
        else hipLaunchKernelGGL((append_rows_kernel<128, true>), grid, block, 0, s, d);
        return hipGetLastError();
    }
    // one unit per wave where possible; every workgroup scans all rows, so
    // the grid shrinks as rows grow (waves then loop over units)
    const int64_t scan_cap = std::max<int64_t>(1024, (int64_t(1) << 22) / (a.num_rows + 1));
    const int64_t wg = std::min<int64_t>((a.n_units + 3) / 4, scan_cap);
    const dim3 grid((unsigned)wg);
    if (head_dim == 64 && !fp8) hipLaunchKernelGGL((append_kernel<64, false>), grid, block, 0, s, a);
    else if (head_dim == 64) hipLaunchKernelGGL((append_kernel<64, true>), grid, block, 0, s, a);
    else if (!fp8) hipLaunchKernelGGL((append_kernel<128, false>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((append_kernel<128, true>), grid, block, 0, s, a);
    return hipGetLastError();
}

hipError_t launch_plan_upload(const void *src, void *dst, int64_t words, hipStream_t s) {
    if (words == 0) return hipSuccess;
    const int64_t wg = std::min<int64_t>((words / 4 + 255) / 256 + 1, 256);
    hipLaunchKernelGGL(plan_upload_kernel, dim3((unsigned)wg), dim3(256), 0, s,
                       (const uint32_t *)src, (uint32_t *)dst, words);
    return hipGetLastError();
}

hipError_t launch_block_copy(const BlockCopyArgs &a, hipStream_t s) {
    if (a.n_pairs == 0) return hipSuccess;
    const dim3 grid((unsigned)((int64_t)a.n_pairs * a.chunks)), block(256);
    hipLaunchKernelGGL(block_copy_kernel, grid, block, 0, s, a);
    return hipGetLastError();
}

int prefill_max_blocks(int head_dim) {
    return (kPfLdsLimit - (head_dim == 64 ? PfLds<64>::BYTES : PfLds<128>::BYTES)) / 4;
}

// The dynamic-LDS limit of kernel f, raised once per device (bit d: done on
// device d; concurrent first calls both set it, which is harmless).
static hipError_t raise_lds_limit(const void *f, std::atomic<uint64_t> &done) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const uint64_t bit = dev >= 0 && dev < 64 ? (1ull << dev) : 0;
    if (!bit || !(done.load(std::memory_order_acquire) & bit)) {
        e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, kPfLdsLimit);
        if (e != hipSuccess) return e;
        done.fetch_or(bit, std::memory_order_release);
    }
    return hipSuccess;
}

template <int D, bool FP8>
static hipError_t launch_prefill_t(const PrefillArgs &p, hipStream_t s) {
    static std::atomic<uint64_t> attr_devices{0};
    hipError_t e = raise_lds_limit((const void *)prefill_kernel<D, FP8>, attr_devices);
    if (e != hipSuccess) return e;
    const int bytes = PfLds<D>::BYTES + 4 * p.max_blocks;
    const dim3 grid((unsigned)(8 * p.per_xcd)), block(kPfThreads);
    hipLaunchKernelGGL((prefill_kernel<D, FP8>), grid, block, bytes, s, p);
    return hipGetLastError();
}

hipError_t launch_prefill(const PrefillArgs &p, int head_dim, bool fp8, hipStream_t s) {
    if (p.n_logical <= 0) return hipSuccess;
    if (head_dim == 64 && !fp8) return launch_prefill_t<64, false>(p, s);
    if (head_dim == 64) return launch_prefill_t<64, true>(p, s);
    if (!fp8) return launch_prefill_t<128, false>(p, s);
    return launch_prefill_t<128, true>(p, s);
}

// Decode launch shape: runs of 16 workgroups, or shorter so that there are
// at least 64 runs, but never shorter than the run length the caller asks
// for in b.run_log2 (at most 32 workgroups); the grid is a multiple of 8 runs
// (logical workgroups past the end exit at once).  Returns the grid size and
// sets b.run_log2.
static int64_t decode_grid(AttnArgs &b) {
    const int64_t nwg = (b.n_waves + 3) / 4;
    const int min_log2 = std::min(std::max(b.run_log2, 0), 5);
    b.run_log2 = 4;
    while (b.run_log2 > 0 && ((int64_t)64 << b.run_log2) > nwg) --b.run_log2;
    b.run_log2 = std::max(b.run_log2, min_log2);
    const int64_t round = (int64_t)8 << b.run_log2;
    return (nwg + round - 1) / round * round;
}

hipError_t launch_decode(const AttnArgs &a, int head_dim, bool fp8, hipStream_t s) {
    if (a.n_waves <= 0) return hipSuccess;
    AttnArgs b = a;
    const dim3 grid((unsigned)decode_grid(b)), block(256);
    if (head_dim == 64 && !fp8) hipLaunchKernelGGL((attn_kernel<64, false>), grid, block, 0, s, b);
    else if (head_dim == 64) hipLaunchKernelGGL((attn_kernel<64, true>), grid, block, 0, s, b);
    else if (!fp8) hipLaunchKernelGGL((attn_kernel<128, false>), grid, block, 0, s, b);
    else hipLaunchKernelGGL((attn_kernel<128, true>), grid, block, 0, s, b);
    return hipGetLastError();
}

hipError_t launch_merge(const MergeArgs &m, int head_dim, hipStream_t s) {
    if (m.n_waves <= 0) return hipSuccess;
    const dim3 grid((unsigned)((m.n_waves + 3) / 4)), block(256);
    if (head_dim == 64) hipLaunchKernelGGL((merge_kernel<64>), grid, block, 0, s, m);
    else hipLaunchKernelGGL((merge_kernel<128>), grid, block, 0, s, m);
    return hipGetLastError();
}

}  // namespace echo
