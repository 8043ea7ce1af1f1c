// y[N] = x[K] . W[K][N] for a 4-bit weight-only quantised W (decode-time
// linear layers of a 4-bit LLM, Sec. 7): x fp16, y fp32, and
//   W[k][n] = (q[k][n] - 8) * s[k / G][n]
// with q the 4-bit code of column n in 32-bit word n / 8 of row k (bits
// 4 (n % 8) .. 4 (n % 8) + 3) and s the fp16 scale of row group k / G.
// Bandwidth-bound: every code byte is read once, 16 bytes per lane per load
// (32 columns of one row).
//
// Arithmetic.  Rows are taken in pairs (k, k+1) of one group.  A byte
// permute puts the same byte of the two rows' words into the low and high
// halves of one register; each half then holds two codes (two columns).  An
// or with an fp16 exponent makes the halves exact fp16 numbers: the low
// nibble under exponent 1024 reads 1024 + q, the high nibble (bits 4..7)
// under exponent 64 reads 64 + q; a packed fp16 subtract of 1032 (resp. 72)
// leaves exactly q - 8 for both rows.  v_dot2_f32_f16 then adds
// x[k] (q[k] - 8) + x[k+1] (q[k+1] - 8) into an fp32 accumulator -- the
// fp16 products are exact in fp32.  Seven VALU instructions per four codes.
//
// Work decomposition.  L lanes span a segment of 32 L columns; the
// workgroup's other lanes are row slots (R = NTHR / L).  Split s of the K
// axis covers whole groups [s gchunk, (s+1) gchunk).  A work item is U
// consecutive row pairs of one group; row slot r takes items r, r + R, ...
// of its split.  An item's codes are summed in fp32 and multiplied by the
// group's scale once, into the lane's running sums (scale is linear, so a
// group split over several items or row slots is still exact up to fp32
// rounding).  Reduction over row slots, waves and splits is fixed-order, as
// in the fp GEMV.
#include "kcommon.h"

namespace nnjit {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));

template <int L, int NTHR, int U, bool VEC>
__global__ void __launch_bounds__(NTHR)
gemv_q4_kernel(GemvQ4Params p)
{
    constexpr int R = NTHR / L;       // row slots per workgroup
    constexpr int NW = NTHR / 64;     // waves
    constexpr int CW = 32 * L;        // columns per workgroup
    static_assert(NTHR % 64 == 0 && 64 % L == 0, "layout");

    const int tid = threadIdx.x;
    const int c = tid % L, rs = tid / L;
    const int seg = blockIdx.x % p.segs, sp = blockIdx.x / p.segs;
    const int n = seg * CW + c * 32;          // first column of this lane
    const int N = p.N, K = p.K, G = p.G;
    const int g0 = sp * p.gchunk;
    const int g1 = min(p.ngroups, g0 + p.gchunk);
    const int P = (G + 1) >> 1;               // row pairs per group
    const int C = (P + U - 1) / U;            // items per group
    const int items = (g1 - g0) * C;
    const int nwords = (N + 7) >> 3;          // words of a row that hold columns < N

    // fp16 exponent patterns, kept in VGPRs so that mask-and-or is one
    // v_and_or_b32 (a VOP3 instruction cannot take two literal constants)
    unsigned mag_lo, mag_hi;
    asm volatile("v_mov_b32 %0, 0x64006400" : "=v"(mag_lo));
    asm volatile("v_mov_b32 %0, 0x54005400" : "=v"(mag_hi));
    const h2 off_lo = {(_Float16)1032.0f, (_Float16)1032.0f};
    const h2 off_hi = {(_Float16)72.0f, (_Float16)72.0f};

    const unsigned *Wq = (const unsigned *)p.Wq;
    const unsigned short *xs = (const unsigned short *)p.x;
    const unsigned short *S = (const unsigned short *)p.S;

    auto codes = [&](int k) -> u32x4 {
        const unsigned *src = Wq + (long long)k * p.ldq + (n >> 3);
        if constexpr (VEC) {
            return *(const u32x4 *)src;
        } else {
            u32x4 v = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if ((n >> 3) + j < nwords) v[j] = src[j];
            return v;
        }
    };

    float acc[32];
#pragma unroll
    for (int e = 0; e < 32; ++e) acc[e] = 0.f;

    if (n < N) {
        for (int t = rs; t < items; t += R) {
            const int gl = t / C;
            const int g = g0 + gl;
            const int i0 = (t - gl * C) * U;
            const int kb = g * G;
            const int ke = (int)min((long long)kb + G, (long long)K);
            // every load of the item first: U row pairs, the pairs' x, the
            // group's 32 scales.  Rows past the group's end are clamped to
            // its last row (in bounds) and meet x = 0.
            u32x4 wa[U], wb[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int ka = kb + 2 * (i0 + u);
                wa[u] = codes(min(ka, ke - 1));
                wb[u] = codes(min(ka + 1, ke - 1));
            }
            unsigned sc[16];
            const unsigned short *srow = S + (long long)g * p.lds + n;
            if constexpr (VEC) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const u32x4 v = *(const u32x4 *)(srow + 8 * j);
#pragma unroll
                    for (int e = 0; e < 4; ++e) sc[4 * j + e] = v[e];
                }
            } else {
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const unsigned lo = (n + 2 * j < N) ? srow[2 * j] : 0u;
                    const unsigned hi = (n + 2 * j + 1 < N) ? srow[2 * j + 1] : 0u;
                    sc[j] = lo | (hi << 16);
                }
            }
            h2 xp[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int ka = kb + 2 * (i0 + u);
                unsigned bits;
                if (p.xpair && ka + 1 < ke) {
                    bits = *(const unsigned *)(xs + ka);    // ka even, x 4-byte aligned
                } else {
                    const unsigned lo = ka < ke ? xs[ka] : 0u;
                    const unsigned hi = ka + 1 < ke ? xs[ka + 1] : 0u;
                    bits = lo | (hi << 16);
                }
                xp[u] = __builtin_bit_cast(h2, bits);
            }

            float ag[32];
#pragma unroll
            for (int e = 0; e < 32; ++e) ag[e] = 0.f;
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int b = 0; b < 4; ++b) {
                        // low half: byte b of row k's word, high half: of row k+1's
                        const unsigned sel = 0x0c000c00u | ((4u + b) << 16) | (unsigned)b;
                        const unsigned tw = __builtin_amdgcn_perm(wb[u][j], wa[u][j], sel);
                        const h2 lo = __builtin_bit_cast(h2, (tw & 0x000F000Fu) | mag_lo) - off_lo;
                        const h2 hi = __builtin_bit_cast(h2, (tw & 0x00F000F0u) | mag_hi) - off_hi;
                        ag[8 * j + 2 * b] = __builtin_amdgcn_fdot2(lo, xp[u], ag[8 * j + 2 * b], false);
                        ag[8 * j + 2 * b + 1] = __builtin_amdgcn_fdot2(hi, xp[u], ag[8 * j + 2 * b + 1], false);
                    }
#pragma unroll
            for (int e = 0; e < 32; ++e) {
                const h2 s2 = __builtin_bit_cast(h2, sc[e >> 1]);
                acc[e] = __builtin_fmaf((float)s2[e & 1], ag[e], acc[e]);
            }
        }
    }

    // 1. row slots inside a wave
#pragma unroll
    for (int off = L; off < 64; off <<= 1)
#pragma unroll
        for (int e = 0; e < 32; ++e) acc[e] += __shfl_xor(acc[e], off, 64);

    // 2. waves of the workgroup, in wave order
    if constexpr (NW > 1) {
        __shared__ float red[NW][L][32];
        const int wave = tid >> 6, lane = tid & 63;
        if (lane < L)
#pragma unroll
            for (int e = 0; e < 32; ++e) red[wave][lane][e] = acc[e];
        __syncthreads();
        if (tid < L) {
#pragma unroll
            for (int e = 0; e < 32; ++e) {
                float v = red[0][tid][e];
#pragma unroll
                for (int w = 1; w < NW; ++w) v += red[w][tid][e];
                acc[e] = v;
            }
        }
    }

    if (tid >= L) return;
    float *dst = p.nsplit == 1 ? p.y : p.ws + (long long)sp * N;
#pragma unroll
    for (int e = 0; e < 32; ++e)
        if (n + e < N) dst[n + e] = acc[e];
}

template <int L, int NTHR, int U, bool VEC>
static hipError_t launch_gemv_q4(const void *params, dim3 grid, hipStream_t stream)
{
    hipLaunchKernelGGL((gemv_q4_kernel<L, NTHR, U, VEC>), grid, dim3(NTHR), 0, stream,
                       *(const GemvQ4Params *)params);
    return hipGetLastError();
}

// Registers: 32 running sums, 32 item sums, U pairs of 16-byte code loads,
// their x pairs, 16 scale words, plus a fixed overhead.  LDS: the cross-wave
// reduction buffer.
constexpr int est_regs_q4(int u) { return 104 + 9 * u; }
constexpr int lds_q4(int nthr, int l) { return nthr > 64 ? (nthr / 64) * l * 32 * 4 : 4; }

// The compiled configurations (L lanes per segment, NTHR threads, U row
// pairs per item, 16-byte loads or word loads).
#define NNJIT_Q4_LIST(X) \
    X(16, 256, 2, true)  \
    X(16, 256, 4, true)  \
    X(16, 256, 8, true)  \
    X(32, 256, 2, true)  \
    X(32, 256, 4, true)  \
    X(32, 256, 8, true)  \
    X(64, 256, 2, true)  \
    X(64, 256, 4, true)  \
    X(64, 256, 8, true)  \
    X(16, 512, 2, true)  \
    X(16, 512, 4, true)  \
    X(16, 512, 8, true)  \
    X(32, 512, 2, true)  \
    X(32, 512, 4, true)  \
    X(16, 1024, 2, true) \
    X(16, 1024, 4, true) \
    X(16, 256, 4, false) \
    X(64, 256, 4, false)

#define NNJIT_Q4_INST(L, NTHR, U, VEC) template __global__ void gemv_q4_kernel<L, NTHR, U, VEC>(GemvQ4Params);
NNJIT_Q4_LIST(NNJIT_Q4_INST)

#if !defined(__HIP_DEVICE_COMPILE__)
#define NNJIT_Q4_ENTRY(L, NTHR, U, VEC)                                                                              \
    {"gemv_q4_L" #L "_t" #NTHR "_u" #U "_v" #VEC, FAM_GEMV_Q4, 0, 0, 1, 32 * L, 2 * (NTHR / L), NTHR / 64, 1, 0, 0, \
     1, (VEC ? 16 : 4), L, U, NTHR, lds_q4(NTHR, L), est_regs_q4(U),                                             \
     (const void *)&gemv_q4_kernel<L, NTHR, U, VEC>, &launch_gemv_q4<L, NTHR, U, VEC>, 0},
const Variant kGemvQ4Variants[] = {NNJIT_Q4_LIST(NNJIT_Q4_ENTRY)};
const int kNumGemvQ4Variants = sizeof(kGemvQ4Variants) / sizeof(kGemvQ4Variants[0]);
#endif

}  // namespace nnjit
