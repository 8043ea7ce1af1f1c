// y[N] = x[K] . W for a 4-bit weight-only quantised W (decode-time linear
// layers of a 4-bit LLM, Sec. 7), W stored as a linear layer's weight: one
// row per output n, eight 4-bit codes per 32-bit word along the inputs k,
// one fp16 scale per output and group of G inputs:
//   W[k][n] = (q[n][k] - 8) * s[n][k / G],  x fp16, y fp32.
// Bandwidth-bound: every code byte is read once, 16 bytes (32 codes) per lane
// per load, a wave's load covering 2048 consecutive inputs of one row.
//
// Work decomposition.  A wave owns RW consecutive output rows; the KS waves
// of a row group split the row's 2048-input blocks between them (block j to
// wave j mod KS).  No output is shared between workgroups: one kernel, no
// partial sums in device memory.  Sums: per lane over its blocks, then across
// the 64 lanes (butterfly), then across the KS waves in wave order (LDS), a
// fixed order, so results are deterministic.
//
// Arithmetic (16-byte configurations, G a multiple of 32, so the 32 codes of
// a lane share one scale).  A word holds inputs k .. k+7 of one row.  Masking
// with 0x000F000F puts the codes of k and k+4 in the low four bits of the two
// fp16 halves; or-ing in the exponent of 1024 makes them the exact fp16
// numbers 1024 + q, and a packed fp16 subtract of 1032 leaves q - 8 exactly.
// Masking with 0x00F000F0 (codes of k+1, k+5 in bits 4..7) under the exponent
// of 64 gives 64 + q, minus 72; a shift by 8 does the same for k+2, k+6 and
// k+3, k+7.  The x values are regrouped once per block into the matching
// pairs (x[k], x[k+4]) ..., shared by the wave's RW rows, and v_dot2_f32_f16
// adds the two products into an fp32 sum.  Per 8 codes: 4 mask-and-or, 1
// shift, 4 packed subtracts, 4 dot2.  Each item's sum times its scale goes
// into the row's running fp32 sum.  (dot2 is exact to about one fp32 ulp for
// normal fp16 operands; with subnormal ones -- codes read as q 2^-24 without
// an exponent -- it was measured to keep only about 14 bits, so the codes are
// always made normal numbers first.)
//
// The word-load configurations (any G, any alignment) take each code through
// fp32: w = (q - 8) s exactly, y += x w.
#include "kcommon.h"

namespace nnjit {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));

constexpr int kQ4Block = 2048;   // inputs per wave load: 64 lanes x 32 codes

template <int RW, int NTHR, int KS, int UB>
__global__ void __launch_bounds__(NTHR)
gemv_q4_kernel(GemvQ4Params p)
{
    constexpr int NW = NTHR / 64;       // waves
    constexpr int RG = NW / KS;         // row groups per workgroup
    static_assert(NTHR % 64 == 0 && NW % KS == 0, "layout");
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int rg = wave / KS, ks = wave - rg * KS;
    const int n0 = (blockIdx.x * RG + rg) * RW;
    const int K = p.K, N = p.N, G = p.G;
    const int nblk = (K + kQ4Block - 1) / kQ4Block;

    const unsigned *wrow[RW];
    const unsigned short *srow[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) {
        const int n = min(n0 + r, N - 1);      // rows past N: read row N - 1, never stored
        wrow[r] = (const unsigned *)p.Wq + (long long)n * p.ldq;
        srow[r] = (const unsigned short *)p.S + (long long)n * p.lds;
    }
    const unsigned short *xs = (const unsigned short *)p.x;
    // fp16 exponent patterns, kept in VGPRs so that mask-and-or is one
    // v_and_or_b32 (a VOP3 instruction cannot take two literal constants)
    unsigned mag_lo, mag_hi;
    asm volatile("v_mov_b32 %0, 0x64006400" : "=v"(mag_lo));
    asm volatile("v_mov_b32 %0, 0x54005400" : "=v"(mag_hi));
    const h2 off_lo = {(_Float16)1032.0f, (_Float16)1032.0f};
    const h2 off_hi = {(_Float16)72.0f, (_Float16)72.0f};

    float acc[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) acc[r] = 0.f;

    const int klast = ((K - 1) >> 5) << 5;       // start of the last 32-input chunk
    for (int j0 = ks; j0 < nblk; j0 += KS * UB) {
        u32x4 wv[UB][RW];
        unsigned sv[UB][RW];
        u32x4 xv[UB][4];
        // every load of UB blocks first.  Codes and scales are read from the
        // chunk clamped into the row (always in bounds); a chunk past the row
        // meets x = 0, so it adds exactly nothing
#pragma unroll
        for (int b = 0; b < UB; ++b) {
            const int j = j0 + b * KS;
            const int k0 = j * kQ4Block + lane * 32;
            const bool live = j < nblk && k0 < K;
            const int kc = min(k0, klast);
#pragma unroll
            for (int r = 0; r < RW; ++r) {
                wv[b][r] = __builtin_nontemporal_load((const u32x4 *)(wrow[r] + (kc >> 3)));
                sv[b][r] = srow[r][kc / G];
            }
            if (live && k0 + 32 <= K) {
#pragma unroll
                for (int m = 0; m < 4; ++m) xv[b][m] = *(const u32x4 *)(xs + k0 + 8 * m);
            } else {
                // the row's last, partial block: inputs at or past K read as +0
#pragma unroll
                for (int m = 0; m < 4; ++m)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int k = k0 + 8 * m + 2 * e;
                        const unsigned lo = (live && k < K) ? xs[k] : 0u;
                        const unsigned hi = (live && k + 1 < K) ? xs[k + 1] : 0u;
                        xv[b][m][e] = lo | (hi << 16);
                    }
            }
        }
#pragma unroll
        for (int b = 0; b < UB; ++b) {
            // x regrouped into the pairs that meet the decoded codes
            h2 xp[4][4];
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const u32x4 d = xv[b][m];       // (x0,x1) (x2,x3) (x4,x5) (x6,x7)
                xp[m][0] = __builtin_bit_cast(h2, __builtin_amdgcn_perm(d[2], d[0], 0x05040100u));  // (x0, x4)
                xp[m][1] = __builtin_bit_cast(h2, __builtin_amdgcn_perm(d[2], d[0], 0x07060302u));  // (x1, x5)
                xp[m][2] = __builtin_bit_cast(h2, __builtin_amdgcn_perm(d[3], d[1], 0x05040100u));  // (x2, x6)
                xp[m][3] = __builtin_bit_cast(h2, __builtin_amdgcn_perm(d[3], d[1], 0x07060302u));  // (x3, x7)
            }
#pragma unroll
            for (int r = 0; r < RW; ++r) {
                float a = 0.f;
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    const unsigned w = wv[b][r][m], t = w >> 8;
                    const h2 q04 = __builtin_bit_cast(h2, (w & 0x000F000Fu) | mag_lo) - off_lo;
                    const h2 q15 = __builtin_bit_cast(h2, (w & 0x00F000F0u) | mag_hi) - off_hi;
                    const h2 q26 = __builtin_bit_cast(h2, (t & 0x000F000Fu) | mag_lo) - off_lo;
                    const h2 q37 = __builtin_bit_cast(h2, (t & 0x00F000F0u) | mag_hi) - off_hi;
                    a = __builtin_amdgcn_fdot2(q04, xp[m][0], a, false);
                    a = __builtin_amdgcn_fdot2(q15, xp[m][1], a, false);
                    a = __builtin_amdgcn_fdot2(q26, xp[m][2], a, false);
                    a = __builtin_amdgcn_fdot2(q37, xp[m][3], a, false);
                }
                const _Float16 s = __builtin_bit_cast(_Float16, (unsigned short)sv[b][r]);
                acc[r] = __builtin_fmaf((float)s, a, acc[r]);
            }
        }
    }

    // across the lanes of the wave
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
#pragma unroll
        for (int r = 0; r < RW; ++r) acc[r] += __shfl_xor(acc[r], off, 64);

    // across the K-slice waves of the row group, in wave order
    if constexpr (KS > 1) {
        __shared__ float red[NW][RW];
        if (lane == 0)
#pragma unroll
            for (int r = 0; r < RW; ++r) red[wave][r] = acc[r];
        __syncthreads();
        if (ks != 0) return;
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            float v = red[wave][r];
#pragma unroll
            for (int w = 1; w < KS; ++w) v += red[wave + w][r];
            acc[r] = v;
        }
    }
    if (lane == 0)
#pragma unroll
        for (int r = 0; r < RW; ++r)
            if (n0 + r < N) p.y[n0 + r] = acc[r];
}

// Word loads: any group size and alignment.  Lane l takes words l, l + 64, ...
// of its rows; each code goes through fp32 with its own group's scale.
template <int RW, int NTHR>
__global__ void __launch_bounds__(NTHR)
gemv_q4_words_kernel(GemvQ4Params p)
{
    constexpr int NW = NTHR / 64;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n0 = (blockIdx.x * NW + wave) * RW;
    const int K = p.K, N = p.N, G = p.G;
    const int nwords = (K + 7) >> 3;
    const unsigned *wrow[RW];
    const unsigned short *srow[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) {
        const int n = min(n0 + r, N - 1);
        wrow[r] = (const unsigned *)p.Wq + (long long)n * p.ldq;
        srow[r] = (const unsigned short *)p.S + (long long)n * p.lds;
    }
    const _Float16 *xh = (const _Float16 *)p.x;
    const _Float16 *sh[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) sh[r] = (const _Float16 *)srow[r];
    float acc[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) acc[r] = 0.f;
    for (int wi = lane; wi < nwords; wi += 64) {
        unsigned wd[RW];
#pragma unroll
        for (int r = 0; r < RW; ++r) wd[r] = wrow[r][wi];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int k = 8 * wi + i;
            if (k < K) {
                const float xk = (float)xh[k];
#pragma unroll
                for (int r = 0; r < RW; ++r) {
                    const float q = (float)((int)((wd[r] >> (4 * i)) & 15u) - 8);
                    acc[r] = __builtin_fmaf(xk, q * (float)sh[r][k / G], acc[r]);
                }
            }
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
#pragma unroll
        for (int r = 0; r < RW; ++r) acc[r] += __shfl_xor(acc[r], off, 64);
    if (lane == 0)
#pragma unroll
        for (int r = 0; r < RW; ++r)
            if (n0 + r < N) p.y[n0 + r] = acc[r];
}

template <int RW, int NTHR, int KS, int UB>
static hipError_t launch_gemv_q4(const void *params, dim3 grid, hipStream_t stream)
{
    hipLaunchKernelGGL((gemv_q4_kernel<RW, NTHR, KS, UB>), grid, dim3(NTHR), 0, stream,
                       *(const GemvQ4Params *)params);
    return hipGetLastError();
}

template <int RW, int NTHR>
static hipError_t launch_gemv_q4_words(const void *params, dim3 grid, hipStream_t stream)
{
    hipLaunchKernelGGL((gemv_q4_words_kernel<RW, NTHR>), grid, dim3(NTHR), 0, stream,
                       *(const GemvQ4Params *)params);
    return hipGetLastError();
}

// Registers: per block in flight, RW code loads (4 words) and scales, the
// block's 16 x words and their 16 regrouped pairs; RW running sums; a fixed
// overhead.  LDS: the cross-wave buffer of K-sliced configurations.
constexpr int est_regs_q4(int rw, int ub) { return ub * (5 * rw + 32) + rw + 24; }
constexpr int lds_q4(int nthr, int rw, int ks) { return ks > 1 ? (nthr / 64) * rw * 4 : 0; }

// The compiled configurations: RW rows per wave, NTHR threads, KS K-slices
// (waves per row group), UB blocks in flight.
#define NNJIT_Q4_LIST(X) \
    X(2, 256, 1, 2)      \
    X(4, 256, 1, 1)      \
    X(4, 256, 1, 2)      \
    X(8, 256, 1, 1)      \
    X(8, 256, 1, 2)      \
    X(2, 256, 2, 2)      \
    X(4, 256, 2, 1)      \
    X(4, 256, 2, 2)      \
    X(8, 256, 2, 1)      \
    X(1, 256, 4, 2)      \
    X(2, 256, 4, 2)      \
    X(4, 256, 4, 1)      \
    X(4, 128, 1, 2)      \
    X(8, 128, 1, 1)      \
    X(4, 64, 1, 2)       \
    X(8, 64, 1, 1)

#define NNJIT_Q4_WORDS_LIST(X) \
    X(1, 256)                  \
    X(4, 256)

#define NNJIT_Q4_INST(RW, NTHR, KS, UB) template __global__ void gemv_q4_kernel<RW, NTHR, KS, UB>(GemvQ4Params);
NNJIT_Q4_LIST(NNJIT_Q4_INST)
#define NNJIT_Q4_WORDS_INST(RW, NTHR) template __global__ void gemv_q4_words_kernel<RW, NTHR>(GemvQ4Params);
NNJIT_Q4_WORDS_LIST(NNJIT_Q4_WORDS_INST)

#if !defined(__HIP_DEVICE_COMPILE__)
// Variant fields: mt = rows per wave, nt = rows per workgroup, kt = inputs per
// wave load, wm = waves, kslices = K-slices, unroll = blocks in flight.
#define NNJIT_Q4_ENTRY(RW, NTHR, KS, UB)                                                                            \
    {"gemv_q4_r" #RW "_t" #NTHR "_k" #KS "_u" #UB, FAM_GEMV_Q4, 0, 0, RW, RW * (NTHR / 64) / KS, kQ4Block,       \
     NTHR / 64, 1, 0, 0, KS, 16, 64, UB, NTHR, lds_q4(NTHR, RW, KS), est_regs_q4(RW, UB),                       \
     (const void *)&gemv_q4_kernel<RW, NTHR, KS, UB>, &launch_gemv_q4<RW, NTHR, KS, UB>, 0, -1, 0},
#define NNJIT_Q4_WORDS_ENTRY(RW, NTHR)                                                                               \
    {"gemv_q4_words_r" #RW "_t" #NTHR, FAM_GEMV_Q4, 0, 0, RW, RW * (NTHR / 64), 512, NTHR / 64, 1, 0, 0, 1, 4, 64, 1, \
     NTHR, 0, 3 * RW + 40, (const void *)&gemv_q4_words_kernel<RW, NTHR>, &launch_gemv_q4_words<RW, NTHR>, 0, -1, 0},
const Variant kGemvQ4Variants[] = {NNJIT_Q4_LIST(NNJIT_Q4_ENTRY) NNJIT_Q4_WORDS_LIST(NNJIT_Q4_WORDS_ENTRY)};
const int kNumGemvQ4Variants = sizeof(kGemvQ4Variants) / sizeof(kGemvQ4Variants[0]);
#endif

}  // namespace nnjit
