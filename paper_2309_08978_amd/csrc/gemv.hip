// y[N] = x[K] . W[K][N] for M == 1 (decode-time linear layers), fp32 or
// fp16 operands, fp32 accumulation and output.  Bandwidth-bound: every byte
// of W is read once, 128 bits per lane per load.
//
// Workgroup layout.  L lanes span one segment of L*V consecutive columns
// (V = 4 fp32 or 8 fp16 columns per 128-bit load); the workgroup's other
// lanes are row slots, so a wave reads 64/L rows of the segment at once and
// the workgroup NTHR/L rows.  Each lane keeps U row loads in flight.  The
// K rows of W are split over S workgroups per segment (split-K).
//
// Reduction over k, in a fixed order (deterministic):
//   1. across the row slots of a wave: butterfly over lane xor L, 2L, ...
//   2. across the waves of the workgroup: through LDS, wave 0 sums in order;
//   3. across the S workgroups of a segment: partials in device memory,
//      summed in split order by a second, elementwise kernel.
#include "kcommon.h"

namespace nnjit {

template <typename T> struct WTraits;
template <> struct WTraits<float> {
    static constexpr int V = 4;
    __device__ static __forceinline__ void fma(float (&acc)[4], float x, u32x4 w) {
        const f32x4 f = __builtin_bit_cast(f32x4, w);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] = __builtin_fmaf(x, f[e], acc[e]);
    }
    __device__ static __forceinline__ float load1(const void *p, long long i) { return ((const float *)p)[i]; }
    __device__ static __forceinline__ unsigned bits1(const void *p, long long i) {
        return __builtin_bit_cast(unsigned, ((const float *)p)[i]);
    }
};
template <> struct WTraits<_Float16> {
    static constexpr int V = 8;
    __device__ static __forceinline__ void fma(float (&acc)[8], float x, u32x4 w) {
        const f16x8 h = __builtin_bit_cast(f16x8, w);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = __builtin_fmaf(x, (float)h[e], acc[e]);
    }
    __device__ static __forceinline__ float load1(const void *p, long long i) {
        return (float)((const _Float16 *)p)[i];
    }
    __device__ static __forceinline__ unsigned bits1(const void *p, long long i) {
        return ((const unsigned short *)p)[i];
    }
};

template <typename T, int L, int NTHR, int U, bool VEC>
__global__ void __launch_bounds__(NTHR)
gemv_kernel(GemvParams p)
{
    typedef WTraits<T> W_;
    constexpr int V = W_::V;
    constexpr int CW = L * V;         // columns per workgroup
    constexpr int R = NTHR / L;       // row slots per workgroup
    constexpr int NW = NTHR / 64;     // waves
    static_assert(NTHR % 64 == 0 && 64 % L == 0, "layout");

    const int tid = threadIdx.x;
    const int c = tid % L, rs = tid / L;
    // consecutive segments on one XCD: narrow segments (L * V * sizeof(T) <
    // 128 bytes) share cache lines with their neighbours, read once into
    // that XCD's L2
    const int logical = xcd_remap(blockIdx.x, gridDim.x);
    const int seg = logical % p.segs, s = logical / p.segs;
    const int n = seg * CW + c * V;
    const int kbeg = s * p.kchunk;
    const int kend = min(p.K, kbeg + p.kchunk);
    const int N = p.N;

    float acc[V];
#pragma unroll
    for (int e = 0; e < V; ++e) acc[e] = 0.f;

    const T *W = (const T *)p.W;
    auto wload = [&](int k) -> u32x4 {
        const T *src = W + (long long)k * p.ldw + n;
        if constexpr (VEC) {
            // W is read exactly once: a non-temporal load
            return __builtin_nontemporal_load((const u32x4 *)src);
        } else {
            // element loads, columns at or beyond N read as +0
            u32x4 v = {0u, 0u, 0u, 0u};
            if constexpr (V == 4) {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (n + e < N) v[e] = W_::bits1(src, e);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (n + e < N) v[e >> 1] |= W_::bits1(src, e) << (16 * (e & 1));
            }
            return v;
        }
    };

    if (n < N) {
        int k = kbeg + rs;
        for (; k + (U - 1) * R < kend; k += U * R) {
            u32x4 w[U];
            float xv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) w[u] = wload(k + u * R);
#pragma unroll
            for (int u = 0; u < U; ++u) xv[u] = W_::load1(p.x, k + u * R);
#pragma unroll
            for (int u = 0; u < U; ++u) W_::fma(acc, xv[u], w[u]);
        }
        for (; k < kend; k += R) W_::fma(acc, W_::load1(p.x, k), wload(k));
    }

    // 1. row slots inside a wave
#pragma unroll
    for (int off = L; off < 64; off <<= 1)
#pragma unroll
        for (int e = 0; e < V; ++e) acc[e] += __shfl_xor(acc[e], off, 64);

    // 2. waves of the workgroup
    if constexpr (NW > 1) {
        __shared__ float red[NW][L][V];
        const int wave = tid >> 6, lane = tid & 63;
        if (lane < L)
#pragma unroll
            for (int e = 0; e < V; ++e) red[wave][lane][e] = acc[e];
        __syncthreads();
        if (tid < L) {
#pragma unroll
            for (int e = 0; e < V; ++e) {
                float v = red[0][tid][e];
#pragma unroll
                for (int w = 1; w < NW; ++w) v += red[w][tid][e];
                acc[e] = v;
            }
        }
    }
    // threads tid < L now hold the workgroup's sums for columns n .. n+V-1

    if (p.S == 1) {
        if (tid < L)
#pragma unroll
            for (int e = 0; e < V; ++e)
                if (n + e < N) p.y[n + e] = acc[e];
        return;
    }

    // 3. split-K: this split's partial row, summed in split order by the
    //    reduction kernel
    if (tid < L)
#pragma unroll
        for (int e = 0; e < V; ++e)
            if (n + e < N) p.ws[(long long)s * N + n + e] = acc[e];
}

template <typename T, int L, int NTHR, int U, bool VEC>
static hipError_t launch_gemv(const void *params, dim3 grid, hipStream_t stream)
{
    hipLaunchKernelGGL((gemv_kernel<T, L, NTHR, U, VEC>), grid, dim3(NTHR), 0, stream,
                       *(const GemvParams *)params);
    return hipGetLastError();
}

// Registers: V accumulators, U in-flight 128-bit loads and their x values,
// plus a fixed overhead.  LDS: the cross-wave reduction buffer.
constexpr int est_regs_gemv(int v, int u) { return v + 5 * u + 24; }
constexpr int lds_gemv(int nthr, int l, int v) { return nthr > 64 ? (nthr / 64) * l * v * 4 + 4 : 4; }

#define NNJIT_GEMV_VARIANT(T, FAMV, V, L, NTHR, U, VEC)                                                 \
    {"gemv_" #T "_L" #L "_t" #NTHR "_u" #U "_v" #VEC, FAMV, 0, 0, 1, L * V, NTHR / L, NTHR / 64, 1, 0, 0, 1, \
     (VEC ? 16 : (int)sizeof(T)), L, U, NTHR, lds_gemv(NTHR, L, V), est_regs_gemv(V, U),                \
     (const void *)&gemv_kernel<T, L, NTHR, U, VEC>, &launch_gemv<T, L, NTHR, U, VEC>, 0, -1, 0}


// The compiled GEMV configurations of both dtypes.
#define NNJIT_GEMV_LIST(X) \
    X(float, 16, 256, 16, true) \
    X(float, 64, 256, 16, true) \
    X(float, 16, 512, 8, true) \
    X(_Float16, 16, 256, 16, true) \
    X(_Float16, 32, 256, 16, true) \
    X(_Float16, 64, 256, 16, true) \
    X(_Float16, 16, 512, 8, true) \
    X(_Float16, 32, 512, 8, true) \
    X(float, 64, 256, 4, true) \
    X(float, 64, 256, 8, true) \
    X(float, 64, 512, 4, true) \
    X(float, 64, 512, 8, true) \
    X(float, 64, 128, 8, true) \
    X(float, 64, 64, 8, true) \
    X(float, 32, 256, 4, true) \
    X(float, 32, 256, 8, true) \
    X(float, 32, 512, 4, true) \
    X(float, 16, 256, 4, true) \
    X(float, 16, 256, 8, true) \
    X(float, 16, 512, 4, true) \
    X(float, 64, 256, 2, true) \
    X(float, 64, 1024, 4, true) \
    X(float, 64, 256, 4, false) \
    X(_Float16, 64, 256, 4, true) \
    X(_Float16, 64, 256, 8, true) \
    X(_Float16, 64, 512, 4, true) \
    X(_Float16, 64, 512, 8, true) \
    X(_Float16, 64, 128, 8, true) \
    X(_Float16, 64, 64, 8, true) \
    X(_Float16, 32, 256, 4, true) \
    X(_Float16, 32, 256, 8, true) \
    X(_Float16, 32, 512, 4, true) \
    X(_Float16, 16, 256, 4, true) \
    X(_Float16, 16, 256, 8, true) \
    X(_Float16, 16, 512, 4, true) \
    X(_Float16, 64, 256, 2, true) \
    X(_Float16, 64, 1024, 4, true) \
    X(_Float16, 64, 256, 4, false) \
    X(_Float16, 8, 256, 8, true) \
    X(_Float16, 8, 512, 8, true) \
    X(_Float16, 8, 512, 4, true) \
    X(_Float16, 8, 1024, 4, true) \
    X(_Float16, 4, 256, 8, true) \
    X(_Float16, 4, 512, 8, true) \
    X(_Float16, 4, 512, 4, true) \
    X(_Float16, 4, 1024, 4, true) \
    X(float, 8, 256, 8, true) \
    X(float, 8, 512, 8, true) \
    X(float, 8, 512, 4, true) \
    X(float, 8, 1024, 4, true) \
    X(float, 4, 512, 8, true) \
    X(float, 8, 1024, 8, true) \
    X(float, 16, 1024, 8, true) \
    X(_Float16, 4, 1024, 8, true) \
    X(_Float16, 8, 1024, 8, true) \
    X(_Float16, 2, 1024, 8, true) \

#define NNJIT_GEMV_INST(T, L, NTHR, U, VEC) template __global__ void gemv_kernel<T, L, NTHR, U, VEC>(GemvParams);
NNJIT_GEMV_LIST(NNJIT_GEMV_INST)

#if !defined(__HIP_DEVICE_COMPILE__)
#define NNJIT_GEMV_ENTRY(T, L, NTHR, U, VEC)                                                                    \
    NNJIT_GEMV_VARIANT(T, (sizeof(T) == 4 ? FAM_GEMV_F32 : FAM_GEMV_F16), (16 / (int)sizeof(T)), L, NTHR, U, VEC),
const Variant kGemvVariants[] = {NNJIT_GEMV_LIST(NNJIT_GEMV_ENTRY)};
const int kNumGemvVariants = sizeof(kGemvVariants) / sizeof(kGemvVariants[0]);
#endif

// ------------------------------------------------------------------------
// Split-K reduction: one thread per 4 consecutive columns of one output row,
// partials summed in split order 0, 1, ..., S-1 (deterministic).  Partials
// are loaded 8 at a time (indices clamped to S-1, so the loads are
// unconditional and all in flight together) and added in order.
__global__ void __launch_bounds__(256)
splitk_reduce_kernel(const float *__restrict__ ws, int S, long long slice, int rows, int M, int N, float *C,
                     long long ldc, long long sC)
{
    const int nq = (N + 3) >> 2;
    const long long total = (long long)rows * nq;
    const long long stride = (long long)gridDim.x * blockDim.x;
    for (long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        const int r = (int)(t / nq), j = (int)(t - (long long)r * nq) * 4;
        const int z = r / M, i = r - z * M;
        const float *src = ws + (long long)r * N + j;
        float *dst = C + z * sC + (long long)i * ldc + j;
        if ((N & 3) == 0) {
            f32x4 v = *(const f32x4 *)src;
            for (int s0 = 1; s0 < S; s0 += 8) {
                f32x4 w[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) w[u] = *(const f32x4 *)(src + min(s0 + u, S - 1) * slice);
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (s0 + u < S)
#pragma unroll
                        for (int e = 0; e < 4; ++e) v[e] += w[u][e];
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) dst[e] = v[e];
        } else {
            for (int e = 0; e < 4 && j + e < N; ++e) {
                float v = src[e];
                for (int s0 = 1; s0 < S; s0 += 8) {
                    float w[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) w[u] = src[min(s0 + u, S - 1) * slice + e];
#pragma unroll
                    for (int u = 0; u < 8; ++u)
                        if (s0 + u < S) v += w[u];
                }
                dst[e] = v;
            }
        }
    }
}

hipError_t launch_splitk_reduce(const float *ws, int S, int batch, int M, int N, float *C, long long ldc,
                                long long sC, hipStream_t stream)
{
    const int rows = batch * M;
    const long long total = (long long)rows * ((N + 3) / 4);
    if (total <= 0) return hipSuccess;
    // small outputs (a GEMV's single row) in 64-thread workgroups, so that
    // their few thousand threads spread over as many CUs as possible
    const int tpb = total < 64LL * 1024 ? 64 : 256;
    long long blocks = (total + tpb - 1) / tpb;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)blocks), dim3(tpb), 0, stream, ws, S,
                       (long long)rows * N, rows, M, N, C, ldc, sC);
    return hipGetLastError();
}

// ------------------------------------------------------------------------
// Stream-K fix-up.  Workgroup w of the GEMM took units [u0(w), u0(w + 1)),
// u0(w) = w units / G.  A tile is shared when a boundary u0(b) (b = 1 .. G-1)
// falls strictly inside it; workgroup b - 1 then holds its first units.
// kFixupParts workgroups here per boundary, each taking a quarter of the
// tile's element quads: those of the first boundary inside a tile sum the
// tile's pieces over the sharing workgroups, in workgroup (= K) order, and
// write the tile of C.  A piece is in slot 2w if the tile is workgroup w's
// first segment, else in slot 2w + 1: every sharing workgroup after b - 1
// starts inside the tile (slot 2w); b - 1 starts at the tile's first unit
// (slot 2(b - 1)) or before it (2(b - 1) + 1).  Each thread keeps QB quads
// times up to 4 pieces of loads in flight before it stores.
constexpr int kFixupThreads = 512, kFixupParts = 4;
__global__ void __launch_bounds__(kFixupThreads)
streamk_fixup_kernel(GemmParams p, int mt, int nt)
{
    constexpr int QB = 4;
    const long long G = p.sk_wgs;
    const int b = blockIdx.x / kFixupParts + 1, part = blockIdx.x % kFixupParts;
    const long long ua = (long long)(b - 1) * p.units / G, ub = (long long)b * p.units / G;
    const long long t = ub / p.nslab;
    const long long tstart = t * p.nslab, tend = tstart + p.nslab;
    if (ub == tstart || ua > tstart) return;   // no shared tile here, or an earlier boundary's
    int nw = 2;                                // sharing workgroups b - 1, b, ...
    while (b - 1 + nw < G && (long long)(b - 1 + nw) * p.units / G < tend) ++nw;
    const long long slot0 = 2LL * (b - 1) + (ua == tstart ? 0 : 1);
    int tm, tn;
    tile_of((int)t, p.tiles_m, p.tiles_n, p.group_m, tm, tn);
    const int m0 = tm * mt, n0 = tn * nt;
    const long long tile_elems = (long long)mt * nt;
    const int quads = mt * nt / 4, nq = nt / 4;
    const int qbeg = (int)((long long)quads * part / kFixupParts);
    const int qend = (int)((long long)quads * (part + 1) / kFixupParts);
    const float *__restrict__ ws = p.ws;
    float *__restrict__ C = p.C;
    const bool vec_c = (p.ldc & 3) == 0 && ((unsigned long long)C & 15) == 0;
    for (int q0 = qbeg + threadIdx.x; q0 < qend; q0 += QB * kFixupThreads) {
        f32x4 acc[QB];
#pragma unroll
        for (int i = 0; i < QB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int w0 = 0; w0 < nw; w0 += 4) {
            f32x4 v[QB][4];   // indices clamped: the loads are unconditional
#pragma unroll
            for (int i = 0; i < QB; ++i)
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int q = min(q0 + i * kFixupThreads, qend - 1), k = min(w0 + u, nw - 1);
                    const long long slot = k == 0 ? slot0 : 2LL * (b - 1 + k);
                    v[i][u] = *(const f32x4 *)(ws + slot * tile_elems + 4LL * q);
                }
#pragma unroll
            for (int i = 0; i < QB; ++i)
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (w0 + u < nw)
#pragma unroll
                        for (int e = 0; e < 4; ++e) acc[i][e] += v[i][u][e];
        }
#pragma unroll
        for (int i = 0; i < QB; ++i) {
            const int q = q0 + i * kFixupThreads;
            if (q >= qend) break;
            const int row = m0 + q / nq, col = n0 + (q % nq) * 4;
            if (row >= p.M) continue;
            float *d = C + (long long)row * p.ldc + col;
            if (vec_c && col + 4 <= p.N) {
                *(f32x4 *)d = acc[i];
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (col + e < p.N) d[e] = acc[i][e];
            }
        }
    }
}

hipError_t launch_streamk_fixup(const GemmParams &p, int mt, int nt, hipStream_t stream)
{
    if (p.sk_wgs < 2) return hipSuccess;
    hipLaunchKernelGGL(streamk_fixup_kernel, dim3((unsigned)((p.sk_wgs - 1) * kFixupParts)), dim3(kFixupThreads), 0,
                       stream, p, mt, nt);
    return hipGetLastError();
}

// ------------------------------------------------------------------------
// Streaming-read reference: every 16-byte chunk of src read once (four loads
// in flight per lane, consecutive lanes on consecutive chunks), combined by
// XOR so the loads cannot be dropped; a workgroup stores only if its value
// hits one constant, so the kernel writes (practically) nothing.  It is the
// measure of what one launch can stream from HBM, set beside the GEMVs.
__global__ void __launch_bounds__(256)
stream_read_kernel(const u32x4 *__restrict__ src, long long n16, unsigned *sink)
{
    const long long stride = (long long)gridDim.x * 256;
    long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    unsigned acc = 0;
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const u32x4 a = __builtin_nontemporal_load(src + i), b = __builtin_nontemporal_load(src + i + stride),
                    c = __builtin_nontemporal_load(src + i + 2 * stride), d = __builtin_nontemporal_load(src + i + 3 * stride);
        acc ^= (a.x ^ a.y ^ a.z ^ a.w) ^ (b.x ^ b.y ^ b.z ^ b.w) ^ (c.x ^ c.y ^ c.z ^ c.w) ^ (d.x ^ d.y ^ d.z ^ d.w);
    }
    for (; i < n16; i += stride) {
        const u32x4 a = __builtin_nontemporal_load(src + i);
        acc ^= a.x ^ a.y ^ a.z ^ a.w;
    }
    if (acc == 0x9e3779b9u) sink[blockIdx.x] = acc;
}

hipError_t launch_stream_read(const void *src, long long bytes, unsigned *sink, int workgroups, hipStream_t stream)
{
    if (bytes <= 0) return hipSuccess;
    hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)workgroups), dim3(256), 0, stream, (const u32x4 *)src,
                       bytes / 16, sink);
    return hipGetLastError();
}

// ------------------------------------------------------------------------
// Scratch fill for the tuner: a counter-based hash of (seed, index) gives
// four uniforms in [-1, 1) per value; their sum, scaled to unit variance
// (times `scale`), is close to normal -- the tuner times candidates on values
// shaped like the workloads' activations and weights, since the matrix cores'
// speed depends somewhat on the data.  FILL_WORDS writes the raw hash.
__device__ __forceinline__ unsigned mix32(unsigned x) {
    x ^= x >> 16; x *= 0x7feb352du; x ^= x >> 15; x *= 0x846ca68bu; x ^= x >> 16;
    return x;
}

__global__ void fill_kernel(void *dst, long long n, int kind, float scale, unsigned seed)
{
    const long long stride = (long long)gridDim.x * blockDim.x;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        unsigned h = mix32((unsigned)i * 0x9e3779b9u ^ mix32(seed + (unsigned)(i >> 32)));
        if (kind == FILL_WORDS) {
            ((unsigned *)dst)[i] = h;
            continue;
        }
        float sum = 0.f;
        for (int u = 0; u < 4; ++u) {
            sum += (float)(h >> 8) * (1.0f / 8388608.0f) - 1.0f;
            h = mix32(h + 0x632be5abu);
        }
        const float v = sum * (0.8660254f * scale);   // sqrt(3)/2: four U[-1,1) have variance 4/3
        if (kind == FILL_F16) ((_Float16 *)dst)[i] = (_Float16)v;
        else ((float *)dst)[i] = v;
    }
}

hipError_t launch_fill(void *dst, long long n, int kind, float scale, unsigned seed, hipStream_t stream)
{
    if (n <= 0) return hipSuccess;
    long long blocks = (n + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, dst, n, kind, scale, seed);
    return hipGetLastError();
}

}  // namespace nnjit
