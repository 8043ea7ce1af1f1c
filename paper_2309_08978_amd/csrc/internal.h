// Internal declarations shared by the kernels, the lite-space builder and
// the runtime of libnnjit.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace nnjit {

// Kernel families.  A family fixes the operand dtype and the kernel template;
// the configurations of a family differ in their tiling parameters.
enum Family { FAM_GEMM_F32 = 0, FAM_GEMM_F16 = 1, FAM_GEMV_F32 = 2, FAM_GEMV_F16 = 3, FAM_GEMV_Q4 = 4, FAM_COUNT = 5 };

// Arguments of the GEMM / BatchMatMul kernels (one product per grid.z slice).
struct GemmParams {
    const void *A;
    const void *B;
    float *C;
    long long lda, ldb, ldc;
    long long sA, sB, sC;  // batch strides, elements
    int M, N, K;
    int batch;             // batch slices in this launch (grid.z)
    int S;                 // split-K factor
    int kchunk;            // K range of one split, a multiple of the K-slab
    int tiles_m, tiles_n;
    int group_m;           // tile rows per group of the tile order (1 .. tiles_m)
    float *ws;             // S > 1: partial products, row-major [S][batch][M][N];
                           // stream-K: partial tiles, [2 * sk_wgs][Mt][Nt]
    const void *zero;      // >= 64 bytes of zeros: the load address of out-of-range elements
    // Stream-K (sk_wgs > 0, batch 1, S 1): the tiles' K slabs form one
    // sequence of `units` = tiles x nslab units, cut evenly over sk_wgs
    // workgroups; workgroup w takes units [w units / sk_wgs, (w + 1) units /
    // sk_wgs).  A tile covered by one workgroup is stored to C; the pieces of
    // a tile covered by several go to partial slots (the workgroup's first
    // piece to slot 2w, its last to 2w + 1) and a fix-up kernel adds them in
    // workgroup order.
    int sk_wgs;
    int nslab;             // K slabs per tile
    long long units;
};

// Arguments of the M == 1 kernels: y[N] = x[K] . W[K][N].
struct GemvParams {
    const void *x;
    const void *W;
    float *y;
    long long ldw;
    int K, N;
    int S;            // split-K factor
    int kchunk;       // rows of W per split
    int segs;         // column segments
    float *ws;        // S > 1: partial rows, [S][N]
};

// Arguments of the 4-bit weight-only GEMV: y[N] = x[K] . W with
// W[k][n] = (q[n][k] - 8) * S[n][k / G]; row n of q packed eight codes per
// 32-bit word along k (low nibble first), S fp16, x fp16, y fp32.
struct GemvQ4Params {
    const void *x;        // fp16 [K]
    const void *Wq;       // uint32 [N][ldq]
    const void *S;        // fp16 [N][lds]
    float *y;             // fp32 [N]
    long long ldq, lds;
    int K, N, G;
};

typedef hipError_t (*LaunchFn)(const void *params, dim3 grid, hipStream_t stream);

// One compiled kernel instantiation (a point of the lite space's parameter
// axes, before the runtime split-K factor is chosen).
struct Variant {
    const char *name;
    int family;
    int mfma_m, mfma_k;   // matrix-core instruction shape (0 for GEMV)
    int mt, nt, kt;       // macro tile (GEMV: mt = 1, nt = columns per WG, kt = rows per pass)
    int wm, wn;           // wave grid of the workgroup (GEMV: wm = waves, wn = 1)
    int stages;           // LDS buffers for the K loop (GEMV 0)
    int prefetch;         // K slabs in flight (in registers, or in LDS for direct-copy variants; GEMV 0)
    int kslices;          // K groups of waves inside a workgroup (GEMM; GEMV 1)
    int vec_bytes;        // bytes per global load of one lane (16, or the element size)
    int lanes_seg;        // GEMV: lanes across one row segment
    int unroll;           // GEMV: row loads in flight per lane
    int threads;          // workgroup size
    int lds_bytes;        // static LDS of one workgroup
    int est_regs;         // VGPR+AGPR estimate per lane (the Table 1 register formula)
    const void *kernel;   // device function (attribute queries)
    LaunchFn launch;
    int direct_copy;      // 1: slabs go global -> LDS by direct copies (staging in LDS, not registers)
    int lds_layout;       // GEMM A slab in LDS: LAYOUT_SWIZZLE, LAYOUT_PAD or LAYOUT_PLAIN (GEMV: -1)
    int rolled;           // GEMM: 1 if the K steps of a slab run as a loop instead of fully unrolled
};

// LDS layouts of a GEMM's A slab: 16-byte chunk index XOR-swizzled by row,
// rows padded by 16 bytes, or plain rows.
enum LdsLayout { LAYOUT_SWIZZLE = 0, LAYOUT_PAD = 1, LAYOUT_PLAIN = 2 };

// Variant tables, one per family (defined in the kernel sources).
extern const Variant kGemmF32Variants[];
extern const int kNumGemmF32Variants;
extern const Variant kGemmF16Variants[];
extern const int kNumGemmF16Variants;
extern const Variant kGemvVariants[];
extern const int kNumGemvVariants;
extern const Variant kGemvQ4Variants[];
extern const int kNumGemvQ4Variants;

// Device helper kernels: the fixed-order split-K reduction
//   C[z][i][j] = ws[0][z][i][j] + ws[1][z][i][j] + ... + ws[S-1][z][i][j]
// (ws row-major [S][batch][M][N], C with leading dim ldc and batch stride sC),
// and the scratch fill of the tuner: n values of about N(0, scale^2) as fp32
// or fp16, or n random 32-bit words.
hipError_t launch_splitk_reduce(const float *ws, int S, int batch, int M, int N, float *C, long long ldc,
                                long long sC, hipStream_t stream);
// Stream-K fix-up: C tile = sum, in workgroup order, of the partial slots
// of every tile that several workgroups share (see GemmParams).
hipError_t launch_streamk_fixup(const GemmParams &p, int mt, int nt, hipStream_t stream);
enum FillKind { FILL_F32 = 0, FILL_F16 = 1, FILL_WORDS = 2 };
// Fixed device scratch of the allocation-free entry point (split-K partials).
constexpr size_t kNoAllocScratchBytes = (size_t)128 << 20;
// Device addresses of the library's static device arrays on the current
// device: that scratch, and 256 bytes of zeros (the load address of
// out-of-range GEMM elements).
hipError_t static_buffer_addresses(void **scratch_ptr, void **zero_ptr);
// Streaming-read reference kernel (bytes % 16 == 0, src 16-byte aligned,
// sink: `workgroups` words).
hipError_t launch_stream_read(const void *src, long long bytes, unsigned *sink, int workgroups, hipStream_t stream);
hipError_t launch_fill(void *dst, long long n, int kind, float scale, unsigned seed, hipStream_t stream);

}  // namespace nnjit
