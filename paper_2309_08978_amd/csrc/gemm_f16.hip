// fp16-input / fp32-accumulate MatMul / BatchMatMul on the gfx950 matrix
// cores (v_mfma_f32_32x32x16_f16, v_mfma_f32_16x16x32_f16).  C is fp32.
//
// Same tile hierarchy as the fp32 kernels (Fig. 10, Table 1 of the paper):
// an Mt x Nt tile per workgroup, a 64-deep K slab staged through LDS, wave
// sub-tiles in accumulator registers, unrolled inner loop, 128-bit loads.
//
// The matrix cores want both operands K-contiguous per lane (8 halves = one
// 128-bit register quad).  A (row-major M x K) already is; B (row-major
// K x N) is transposed on its way into LDS: each thread loads an 8 x 8 block
// of B (eight 128-bit rows), transposes it in registers and stores eight
// 128-bit columns.  Both LDS slabs are [row][8 chunks of 16 bytes] with the
// chunk index XOR-swizzled by (row >> 1) & 7.  Measured on gfx950: a 128-bit
// LDS read is served 16 lanes (256 bytes) at a time, a 128-bit write 8 lanes
// (128 bytes) at a time.  16 consecutive rows read at one logical chunk then
// hit 16 distinct 16-byte bank groups, and the loaders' stores (8 lanes fill
// the 8 chunks of one row) are conflict-free too, without padding.
#include "kcommon.h"

namespace nnjit {

template <int MF> struct Mfma16;
template <> struct Mfma16<32> {
    typedef f32x16 acc_t;
    static constexpr int NR = 16;
    __device__ static __forceinline__ acc_t mma(f16x8 a, f16x8 b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
    }
    __device__ static __forceinline__ int row_of(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }
};
template <> struct Mfma16<16> {
    typedef f32x4 acc_t;
    static constexpr int NR = 4;
    __device__ static __forceinline__ acc_t mma(f16x8 a, f16x8 b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
    __device__ static __forceinline__ int row_of(int r, int g) { return 4 * g + r; }
};

// Low (even) or high (odd) halves of two dwords, packed low | high << 16.
__device__ __forceinline__ unsigned pack_lo(unsigned a, unsigned b) { return (a & 0xffffu) | (b << 16); }
__device__ __forceinline__ unsigned pack_hi(unsigned a, unsigned b) { return (a >> 16) | (b & 0xffff0000u); }

template <int MT, int NT, int WM, int WN, int MF, int ST, int PF, bool VEC>
__global__ void __launch_bounds__(WM * WN * 64)
gemm_f16_kernel(GemmParams p)
{
    typedef Mfma16<MF> I;
    typedef typename I::acc_t acc_t;
    constexpr int KT = 64;
    constexpr int NTHR = WM * WN * 64;
    constexpr int WTM = MT / WM, WTN = NT / WN;
    constexpr int FM = WTM / MF, FN = WTN / MF;
    constexpr int A8 = MT * (KT / 8);          // 16-byte chunks of the A slab
    constexpr int BB = (KT / 8) * (NT / 8);    // 8x8 blocks of the B slab
    constexpr int LA = (A8 + NTHR - 1) / NTHR;
    constexpr int LB = (BB + NTHR - 1) / NTHR;
    constexpr int KG = 64 / MF;                // lane groups along k (2 or 4)
    constexpr int NSTEP = KT / (8 * KG);       // instructions per slab and fragment pair
    static_assert(FM >= 1 && FN >= 1 && WTM % MF == 0 && WTN % MF == 0, "wave tile");
    static_assert(MT * NT == NTHR * FM * FN * I::NR, "tile / accumulator count");

    __shared__ u32x4 As[ST][MT * 8];
    __shared__ u32x4 Bt[ST][NT * 8];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int li = lane % MF, lg = lane / MF;

    const int tiles = p.tiles_m * p.tiles_n;
    const int gx = gridDim.x;
    const int logical = xcd_remap(blockIdx.x + gx * blockIdx.z, gx * gridDim.z);
    const int z = logical / gx;
    const int rest = logical - z * gx;
    const int s = rest / tiles;
    const int tile = rest - s * tiles;
    int tm, tn;
    tile_of(tile, p.tiles_m, p.tiles_n, p.group_m, tm, tn);
    const int m0 = tm * MT, n0 = tn * NT;
    const int kbeg = s * p.kchunk;
    const int kend = min(p.K, kbeg + p.kchunk);
    const int nk = kend > kbeg ? (kend - kbeg + KT - 1) / KT : 0;

    const unsigned short *A = (const unsigned short *)p.A + (long long)z * p.sA;
    const unsigned short *B = (const unsigned short *)p.B + (long long)z * p.sB;
    float *C = p.C + (long long)z * p.sC;
    const int M = p.M, N = p.N;
    const long long lda = p.lda, ldb = p.ldb;

    // PF slabs in flight in registers (see the fp32 kernel)
    u32x4 ra[PF][LA];
    u32x4 rb[PF][LB][8];

    // 8 halves row[c .. c+7]; elements at or beyond lim, and whole chunks
    // with okr false, are read from the zero buffer (address select only,
    // see the fp32 kernel).
    const unsigned short *zero = (const unsigned short *)p.zero;
    auto ld8 = [&](const unsigned short *row, int c, int lim, bool okr) -> u32x4 {
        u32x4 v;
        if constexpr (VEC) {
            v = *(const u32x4 *)((okr && c < lim) ? row + c : zero);
        } else {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const unsigned lo = *((okr && c + 2 * w < lim) ? row + c + 2 * w : zero);
                const unsigned hi = *((okr && c + 2 * w + 1 < lim) ? row + c + 2 * w + 1 : zero);
                v[w] = lo | (hi << 16);
            }
        }
        return v;
    };

    auto gload = [&](int set, int k0) {
#pragma unroll
        for (int l = 0; l < LA; ++l) {
            const int f = tid + l * NTHR;
            const int row = f >> 3, c = f & 7;
            const int gm = m0 + row;
            const bool okr = (A8 % NTHR == 0 || f < A8) && gm < M;
            ra[set][l] = ld8(A + (long long)gm * lda, k0 + 8 * c, kend, okr);
        }
#pragma unroll
        for (int l = 0; l < LB; ++l) {
            const int f = tid + l * NTHR;
            const int kb = f & 7, nb = f >> 3;
            const int gn = n0 + 8 * nb;
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                const int gk = k0 + 8 * kb + r;
                const bool okr = (BB % NTHR == 0 || f < BB) && gk < kend;
                rb[set][l][r] = ld8(B + (long long)gk * ldb, gn, N, okr);
            }
        }
    };

    auto sstore = [&](int set, int buf) {
#pragma unroll
        for (int l = 0; l < LA; ++l) {
            const int f = tid + l * NTHR;
            if (A8 % NTHR == 0 || f < A8) {
                const int row = f >> 3, c = f & 7;
                As[buf][row * 8 + (c ^ ((row >> 1) & 7))] = ra[set][l];
            }
        }
#pragma unroll
        for (int l = 0; l < LB; ++l) {
            const int f = tid + l * NTHR;
            if (BB % NTHR == 0 || f < BB) {
                const int kb = f & 7, nb = f >> 3;
                // column c of the 8x8 block: halves k = 0..7 of column n = 8*nb + c;
                // the 8 lanes of one LDS write phase fill the 8 chunks of one row
#pragma unroll
                for (int c = 0; c < 8; ++c) {
                    const int d = c >> 1;
                    u32x4 o;
#pragma unroll
                    for (int w = 0; w < 4; ++w)
                        o[w] = (c & 1) ? pack_hi(rb[set][l][2 * w][d], rb[set][l][2 * w + 1][d])
                                       : pack_lo(rb[set][l][2 * w][d], rb[set][l][2 * w + 1][d]);
                    const int n = 8 * nb + c;
                    Bt[buf][n * 8 + (kb ^ ((n >> 1) & 7))] = o;
                }
            }
        }
    };

    acc_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < I::NR; ++r) acc[i][j][r] = 0.f;

    auto compute = [&](int buf) {
#pragma unroll
        for (int st = 0; st < NSTEP; ++st) {
            const int chunk = st * KG + lg;   // k in [8*chunk, 8*chunk + 8)
            f16x8 a[FM], b[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int row = wm * WTM + i * MF + li;
                a[i] = __builtin_bit_cast(f16x8, As[buf][row * 8 + (chunk ^ ((row >> 1) & 7))]);
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int col = wn * WTN + j * MF + li;
                b[j] = __builtin_bit_cast(f16x8, Bt[buf][col * 8 + (chunk ^ ((col >> 1) & 7))]);
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = I::mma(a[i], b[j], acc[i][j]);
        }
    };

    // Software pipeline.  Slab `it` is loaded into staging set it % PF at
    // iteration it - PF, stored to LDS buffer it & 1 at iteration it - 1 and
    // multiplied at iteration it.  The loop is unrolled by PF so every set
    // index is a compile-time constant, and its loads and LDS stores are
    // unconditional (slabs past the end read the zero buffer) so the
    // compiler can keep PF slabs in flight; only the matrix-core work is
    // skipped past the end.
    if (nk > 0) {
#pragma unroll
        for (int u = 0; u < PF; ++u) gload(u, kbeg + u * KT);
        if constexpr (ST == 2) {
            sstore(0, 0);
            __syncthreads();
        }
        for (int it0 = 0; it0 < nk; it0 += PF) {
#pragma unroll
            for (int u = 0; u < PF; ++u) {
                const int it = it0 + u;
                if constexpr (ST == 2) {
                    gload(u, kbeg + (it + PF) * KT);
                    if (it < nk) compute(it & 1);
                    sstore((u + 1) % PF, (it + 1) & 1);
                    __syncthreads();
                } else {
                    __syncthreads();
                    sstore(u, 0);
                    __syncthreads();
                    gload(u, kbeg + (it + PF) * KT);
                    if (it < nk) compute(0);
                }
            }
        }
    }

    const int rbase = m0 + wm * WTM, cbase = n0 + wn * WTN + li;
    if (p.S == 1) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int r = 0; r < I::NR; ++r) {
                    const int row = rbase + i * MF + I::row_of(r, lg), col = cbase + j * MF;
                    if (row < M && col < N) C[(long long)row * p.ldc + col] = acc[i][j][r];
                }
        return;
    }

    // split-K: this split's partial tile goes to ws[s][z][row][col]; a
    // separate kernel sums the S partials in split order
    float *part = p.ws + ((long long)s * p.batch + z) * (long long)M * N;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < I::NR; ++r) {
                const int row = rbase + i * MF + I::row_of(r, lg), col = cbase + j * MF;
                if (row < M && col < N) part[(long long)row * N + col] = acc[i][j][r];
            }
}

template <int MT, int NT, int WM, int WN, int MF, int ST, int PF, bool VEC>
static hipError_t launch_gemm_f16(const void *params, dim3 grid, hipStream_t stream)
{
    hipLaunchKernelGGL((gemm_f16_kernel<MT, NT, WM, WN, MF, ST, PF, VEC>), grid, dim3(WM * WN * 64), 0, stream,
                       *(const GemmParams *)params);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Direct-copy variant ("gemm_f16t").  Both slabs go from global memory to LDS
// with global_load_lds_dwordx4 (no staging registers, no LDS store
// instructions): one such instruction moves 64 x 16 bytes and writes them to
// LDS contiguously at a wave-uniform base, lane l at base + 16 l.  The LDS
// layouts are therefore chosen by which global 16-byte chunk each lane
// fetches.
//
// A slab: [Mt rows][Kt halves], chunk c of row r stored at slot c ^ ((r >> 1)
//   & 7) for 128-byte rows (the conflict-free layout of the kernel above),
//   c ^ ((r >> 2) & 3) for 64-byte rows.
// B slab: row-major [Kt k rows][Nt halves], the 32-byte unit u of row k
//   stored at unit u ^ sB(k), sB(k) = ((k & 3) << 1) | ((k >> 3) & 1).
//
// B is read with ds_read_b64_tr_b16.  Measured on gfx950: within each group
// of 16 lanes, lanes 4r .. 4r+3 each name 8 bytes of a 16-half row r, and
// lane i of the group receives column i of that 4 x 16 block (4 halves, one
// per row).  Naming rows k .. k+3 of the slab at columns n .. n+15 gives lane
// i the halves B[k .. k+3][n + i]: the K-contiguous fragment the matrix core
// wants, without a transpose anywhere.  Two such reads make the 8 halves of
// one fragment.  sB keeps the 4 rows of a group, and the two groups of a
// half-wave (next 16 columns, or next 8 k rows), on distinct banks.
//
// Pipeline: ST LDS stages; slab kk is copied into stage kk % ST while slab
// kk - ST + 1 is multiplied; one barrier per slab.
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;

// Scheduling pattern for NMMA matrix-core instructions and NRD LDS reads of
// one K step: MFMA, reads, MFMA, reads, ... with the reads spread evenly.
template <int Q, int NMMA, int NRD>
__device__ __forceinline__ void interleave_mfma_ds()
{
    if constexpr (Q < NMMA) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
        constexpr int nr = (NRD * (Q + 1)) / NMMA - (NRD * Q) / NMMA;
        if constexpr (nr > 0) __builtin_amdgcn_sched_group_barrier(0x100, nr, 0);   // LDS reads
        interleave_mfma_ds<Q + 1, NMMA, NRD>();
    }
}

template <int MT, int NT, int KT, int WM, int WN, int MF, int ST>
__global__ void __launch_bounds__(WM * WN * 64)
gemm_f16t_kernel(GemmParams p)
{
    typedef Mfma16<MF> I;
    typedef typename I::acc_t acc_t;
    static_assert(KT == 32 || KT == 64, "K slab of 32 or 64 halves");
    constexpr int A_ROW = KT * 2;               // bytes of one A row of the slab
    constexpr int ACH = KT / 8;                 // 16-byte chunks per A row
    constexpr int NW = WM * WN;
    constexpr int WTM = MT / WM, WTN = NT / WN;
    constexpr int FM = WTM / MF, FN = WTN / MF;
    constexpr int KG = 64 / MF;                 // lane groups along k
    constexpr int NSTEP = KT / (8 * KG);        // instructions per slab and fragment pair
    constexpr int A_BYTES = MT * A_ROW;
    constexpr int B_ROW = NT * 2;
    constexpr int B_BYTES = KT * B_ROW;
    constexpr int STAGE = A_BYTES + B_BYTES;
    constexpr int LA = A_BYTES / 1024 / NW, LB = B_BYTES / 1024 / NW;   // copies per wave and slab
    static_assert(LA * NW * 1024 == A_BYTES && LB * NW * 1024 == B_BYTES, "copies must split evenly over waves");
    static_assert(NT >= 128 && (NT & (NT - 1)) == 0, "B swizzle needs a power-of-two row of >= 8 units");
    static_assert(FM >= 1 && FN >= 1 && WTM % MF == 0 && WTN % MF == 0, "wave tile");
    static_assert((ST - 2) * (LA + LB) <= 63, "copies in flight exceed the vmcnt range");

    // A slab swizzle: the 16-byte chunk c of row r sits at c ^ a_swz(r), so
    // that 16 consecutive rows read at one chunk hit distinct bank groups
    // (128-byte rows: (r >> 1) & 7; 64-byte rows: (r >> 2) & 3)
    auto a_swz = [](int row) { return KT == 64 ? ((row >> 1) & 7) : ((row >> 2) & 3); };

    __shared__ __attribute__((aligned(1024))) char smem[ST * STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;

    const int tiles = p.tiles_m * p.tiles_n;
    const int gx = gridDim.x;
    const int logical = xcd_remap(blockIdx.x + gx * blockIdx.z, gx * gridDim.z);
    const int z = logical / gx;
    const int rest = logical - z * gx;
    const int s = rest / tiles;
    const int tile = rest - s * tiles;
    int tm, tn;
    tile_of(tile, p.tiles_m, p.tiles_n, p.group_m, tm, tn);
    const int m0 = tm * MT, n0 = tn * NT;
    const int kbeg = s * p.kchunk;
    const int kend = min(p.K, kbeg + p.kchunk);
    const int nk = kend > kbeg ? (kend - kbeg + KT - 1) / KT : 0;

    const unsigned short *A = (const unsigned short *)p.A + (long long)z * p.sA;
    const unsigned short *B = (const unsigned short *)p.B + (long long)z * p.sB;
    float *C = p.C + (long long)z * p.sC;
    const int M = p.M, N = p.N;
    const long long lda = p.lda, ldb = p.ldb;
    const unsigned short *zero = (const unsigned short *)p.zero;
    typedef __attribute__((address_space(3))) char lds_char;
    auto stage_base = [&](int u) -> lds_char * { return (lds_char *)smem + u * STAGE; };
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);

    // per-lane sources of this wave's copies for the split's first slab;
    // slab kk adds a uniform offset (kk * 64 columns of A, kk * 64 rows of B)
    const unsigned short *a_src[LA];
    int a_k[LA];
    bool a_ok[LA];
#pragma unroll
    for (int j = 0; j < LA; ++j) {
        const int row = (1024 / A_ROW) * (wave + j * NW) + lane / ACH;
        const int col = 8 * ((lane % ACH) ^ a_swz(row));
        a_ok[j] = m0 + row < M;
        a_k[j] = kbeg + col;
        a_src[j] = A + (long long)(a_ok[j] ? m0 + row : 0) * lda + kbeg + col;
    }
    const unsigned short *b_src[LB];
    int b_k[LB];
    bool b_ok[LB];
#pragma unroll
    for (int j = 0; j < LB; ++j) {
        const int o = 1024 * (wave + j * NW) + 16 * lane;
        const int k = o / B_ROW, pos = (o % B_ROW) >> 4;
        const int sb = ((k & 3) << 1) | ((k >> 3) & 1);
        const int col = 16 * ((pos >> 1) ^ sb) + 8 * (pos & 1);
        b_ok[j] = n0 + col < N;
        b_k[j] = kbeg + k;
        b_src[j] = B + (long long)(kbeg + k) * ldb + (b_ok[j] ? n0 + col : 0);
    }

    auto copy_slab = [&](int stage, int kk) {
        const bool live = kk < nk;
        const int dk = kk * KT;
        const long long db = (long long)dk * ldb;
#pragma unroll
        for (int j = 0; j < LA; ++j) {
            const bool ok = live && a_ok[j] && a_k[j] + dk < kend;
            copy16_to_lds(ok ? a_src[j] + dk : zero, (unsigned)(uintptr_t)(stage_base(stage) + 1024 * (wave_u + j * NW)));
        }
#pragma unroll
        for (int j = 0; j < LB; ++j) {
            const bool ok = live && b_ok[j] && b_k[j] + dk < kend;
            copy16_to_lds(ok ? b_src[j] + db : zero,
                          (unsigned)(uintptr_t)(stage_base(stage) + A_BYTES + 1024 * (wave_u + j * NW)));
        }
    };
    // the same copies for a slab that lies wholly inside [kbeg, kend): no
    // checks (rows past M and columns past N were pointed at row / column 0
    // above; what they bring reaches only outputs that are never stored)
    auto copy_full = [&](int stage, int kk) {
        const int dk = kk * KT;
        const long long db = (long long)dk * ldb;
#pragma unroll
        for (int j = 0; j < LA; ++j) {
            copy16_to_lds(a_src[j] + dk, (unsigned)(uintptr_t)(stage_base(stage) + 1024 * (wave_u + j * NW)));
        }
#pragma unroll
        for (int j = 0; j < LB; ++j) {
            copy16_to_lds(b_src[j] + db,
                          (unsigned)(uintptr_t)(stage_base(stage) + A_BYTES + 1024 * (wave_u + j * NW)));
        }
    };
    const int nfull = kend > kbeg ? (kend - kbeg) / KT : 0;   // whole slabs of the range

    acc_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < I::NR; ++r) acc[i][j][r] = 0.f;

    // lane constants of the fragment reads
    const int li = lane % MF, lg = lane / MF;
    const int grp = lane >> 4, tr_r = (lane >> 2) & 3, tr_q = lane & 3;
    const int tr_g = MF == 32 ? grp >> 1 : grp;              // k lane group of this 16-lane group
    const int tr_n = (MF == 32 ? 16 * (grp & 1) : 0) + 4 * tr_q;

    // fragments of one K step (FM A fragments, FN B fragments)
    auto read_frags = [&](lds_char *sa, int st, f16x8 (&a)[FM], f16x8 (&b)[FN]) {
        lds_char *sbp = sa + A_BYTES;
        const int chunk = st * KG + lg;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int row = wm * WTM + i * MF + li;
            a[i] = __builtin_bit_cast(f16x8, *(lds_u32x4 *)(sa + row * A_ROW + 16 * (chunk ^ a_swz(row))));
        }
        const int kc = st * KG + tr_g;                       // 8-row k chunk of this lane group
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int n = wn * WTN + j * MF + tr_n;
            s16x4 h[2];
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
                const int k = 8 * kc + 4 * hh + tr_r;
                const int unit = (n >> 4) ^ ((tr_r << 1) | (kc & 1));
                h[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(sbp + k * B_ROW + unit * 32 + (n & 15) * 2));
            }
            b[j] = __builtin_bit_cast(f16x8, __builtin_shufflevector(h[0], h[1], 0, 1, 2, 3, 4, 5, 6, 7));
        }
    };

    // One slab: the fragments of step st + 1 are read while the matrix
    // cores work on step st, and the scheduler is told to interleave the
    // two (one MFMA, then a share of the LDS reads), so that a wave's own
    // MFMAs cover its LDS latency.
    constexpr int NMMA = FM * FN, NRD = FM + 2 * FN;
    auto compute = [&](int stage) {
        lds_char *sa = stage_base(stage);
        f16x8 a[2][FM], b[2][FN];
        read_frags(sa, 0, a[0], b[0]);
#pragma unroll
        for (int st = 0; st < NSTEP; ++st) {
            const int cur = st & 1;
            if (st + 1 < NSTEP) read_frags(sa, st + 1, a[cur ^ 1], b[cur ^ 1]);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = I::mma(a[cur][i], b[cur][j], acc[i][j]);
            if (st + 1 < NSTEP) interleave_mfma_ds<0, NMMA, NRD>();
        }
    };
    // the same with the first step's fragments passed in (ca, cb); the last
    // step reads the first step of the slab in stage `next` into them, so no
    // slab starts with an LDS wait
    auto compute_carry = [&](int stage, int next, f16x8 (&ca)[FM], f16x8 (&cb)[FN]) {
        lds_char *sa = stage_base(stage);
        f16x8 a[2][FM], b[2][FN];
#pragma unroll
        for (int i = 0; i < FM; ++i) a[0][i] = ca[i];
#pragma unroll
        for (int j = 0; j < FN; ++j) b[0][j] = cb[j];
#pragma unroll
        for (int st = 0; st < NSTEP; ++st) {
            const int cur = st & 1;
            if (st + 1 < NSTEP) read_frags(sa, st + 1, a[cur ^ 1], b[cur ^ 1]);
            else read_frags(stage_base(next), 0, ca, cb);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = I::mma(a[cur][i], b[cur][j], acc[i][j]);
            interleave_mfma_ds<0, NMMA, NRD>();
        }
    };

#pragma unroll
    for (int u = 0; u < ST - 1; ++u) copy_slab(u, u);
    // ST slabs at a time.  While every slab copied in a group is whole (and
    // so is every slab multiplied), the group is one branch-free block with
    // unchecked copies that the scheduler can place among the MFMAs; the
    // rest runs with checked copies and a guard per slab.  Both issue the
    // same copies per slab, so the counted waits are the same.
    int it0 = 0;
    if constexpr (ST >= 4) {
        // With four or more stages the main part runs one slab ahead: the
        // wait and barrier at iteration it make slab it + 1 visible, so the
        // last step of slab it can read slab it + 1's first fragments (one
        // slab fewer of copies in flight, ST - 3)
        if (2 * ST - 1 <= nfull) {
            f16x8 ca[FM], cb[FN];
            wait_vmcnt<(ST - 2) * (LA + LB)>();   // slab 0
            lds_barrier();
            read_frags(stage_base(0), 0, ca, cb);
            for (; it0 + 2 * ST - 1 <= nfull; it0 += ST) {
#pragma unroll
                for (int u = 0; u < ST; ++u) {
                    // this wave's copies of slab it0 + u + 1 are done once
                    // at most the copies of the ST - 3 slabs after it are
                    // pending; the barrier makes every wave's copies visible
                    // and frees the stage of slab it0 + u - 1, whose reads
                    // were issued in the two previous iterations
                    wait_vmcnt<(ST - 3) * (LA + LB)>();
                    lds_barrier();
                    copy_full((u + ST - 1) % ST, it0 + u + ST - 1);
                    compute_carry(u, (u + 1) % ST, ca, cb);
                }
            }
            // the first fragments of slab it0 read by the last iteration go
            // unused: the loop below reads every slab it multiplies itself
        }
    } else {
        for (; it0 + 2 * ST - 1 <= nfull; it0 += ST) {
#pragma unroll
            for (int u = 0; u < ST; ++u) {
                // this wave's copies of slab it0 + u are done once at most
                // the copies of the ST - 2 later slabs are pending; the
                // barrier then makes every wave's copies visible and frees
                // the stage multiplied in the previous iteration
                wait_vmcnt<(ST - 2) * (LA + LB)>();
                lds_barrier();
                copy_full((u + ST - 1) % ST, it0 + u + ST - 1);
                compute(u);
            }
        }
    }
    for (; it0 < nk; it0 += ST) {
#pragma unroll
        for (int u = 0; u < ST; ++u) {
            const int it = it0 + u;
            wait_vmcnt<(ST - 2) * (LA + LB)>();
            lds_barrier();
            copy_slab((u + ST - 1) % ST, it + ST - 1);
            if (it < nk) compute(u);
        }
    }
    wait_vmcnt<0>();   // no copy may still target LDS when the workgroup ends

    const int rbase = m0 + wm * WTM, cbase = n0 + wn * WTN + li;
    float *out = C;
    long long ldo = p.ldc;
    if (p.S > 1) {
        out = p.ws + ((long long)s * p.batch + z) * (long long)M * N;
        ldo = N;
    }
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < I::NR; ++r) {
                const int row = rbase + i * MF + I::row_of(r, lg), col = cbase + j * MF;
                if (row < M && col < N) out[(long long)row * ldo + col] = acc[i][j][r];
            }
}

template <int MT, int NT, int KT, int WM, int WN, int MF, int ST>
static hipError_t launch_gemm_f16t(const void *params, dim3 grid, hipStream_t stream)
{
    hipLaunchKernelGGL((gemm_f16t_kernel<MT, NT, KT, WM, WN, MF, ST>), grid, dim3(WM * WN * 64), 0, stream,
                       *(const GemmParams *)params);
    return hipGetLastError();
}

// Table 1 register formula for one lane (see est_regs_f32): accumulators,
// one K step of A and B fragments (4 VGPRs per 8 halves), the staging
// registers of the global->LDS copy (B needs eight 128-bit rows per 8x8
// block), and a fixed overhead.
constexpr int est_regs_f16(int mt, int nt, int wm, int wn, int mf, int pf) {
    return (mt / wm) * (nt / wn) / 64 + 4 * ((mt / wm) / mf) + 4 * ((nt / wn) / mf) +
           pf * (4 * ((mt * 8 + wm * wn * 64 - 1) / (wm * wn * 64)) +
                 32 * ((nt + wm * wn * 64 - 1) / (wm * wn * 64))) + 28;
}
constexpr int lds_f16(int mt, int nt, int st) { return st * (mt + nt) * 128; }

#define NNJIT_F16_VARIANT(MT, NT, WM, WN, MF, ST, PF, VEC)                                                  \
    {"gemm_f16_" #MT "x" #NT "x64_w" #WM "x" #WN "_m" #MF "_s" #ST "_p" #PF "_v" #VEC, FAM_GEMM_F16, MF,        \
     (MF == 32 ? 16 : 32), MT, NT, 64, WM, WN, ST, PF, 1, (VEC ? 16 : 2), 0, 0, WM * WN * 64,                 \
     lds_f16(MT, NT, ST), est_regs_f16(MT, NT, WM, WN, MF, PF),                                                \
     (const void *)&gemm_f16_kernel<MT, NT, WM, WN, MF, ST, PF, VEC>, &launch_gemm_f16<MT, NT, WM, WN, MF, ST, PF, VEC>, \
     0, LAYOUT_SWIZZLE, 0}

// The compiled fp16 configurations (K slab fixed at 64: 128-byte rows).
#define NNJIT_F16_LIST(X) \
    X(256, 256, 2, 2, 32, 2, 1, true) \
    X(256, 128, 2, 2, 32, 2, 1, true) \
    X(128, 256, 2, 2, 32, 2, 1, true) \
    X(256, 128, 4, 2, 32, 2, 1, true) \
    X(256, 128, 4, 2, 32, 2, 2, true) \
    X(128, 256, 2, 4, 32, 2, 1, true) \
    X(128, 128, 2, 2, 32, 2, 1, true) \
    X(128, 128, 2, 2, 32, 2, 2, true) \
    X(128, 128, 1, 2, 32, 2, 1, true) \
    X(128, 128, 2, 1, 32, 2, 1, true) \
    X(128, 128, 2, 2, 16, 2, 1, true) \
    X(128, 128, 2, 2, 32, 1, 1, true) \
    X(128, 128, 2, 2, 32, 1, 2, true) \
    X(128, 64, 2, 1, 32, 2, 1, true) \
    X(128, 64, 2, 2, 32, 2, 1, true) \
    X(128, 64, 2, 2, 32, 2, 2, true) \
    X(64, 128, 1, 2, 32, 2, 1, true) \
    X(64, 128, 2, 2, 32, 2, 1, true) \
    X(64, 128, 2, 2, 32, 2, 2, true) \
    X(64, 64, 1, 1, 32, 2, 1, true) \
    X(64, 64, 2, 2, 32, 2, 1, true) \
    X(64, 64, 2, 2, 32, 2, 2, true) \
    X(64, 64, 2, 2, 16, 2, 2, true) \
    X(32, 64, 1, 2, 32, 2, 2, true) \
    X(64, 32, 2, 1, 32, 2, 2, true) \
    X(32, 32, 1, 1, 32, 2, 2, true) \
    X(32, 32, 2, 2, 16, 2, 2, true) \
    X(16, 64, 1, 4, 16, 2, 2, true) \
    X(64, 64, 2, 2, 32, 2, 1, false) \
    X(32, 32, 1, 1, 32, 2, 1, false)

// Direct-copy family: accumulators, one K step of fragments, the per-lane
// copy geometry (2 registers per copy) and a fixed overhead; no staging.
constexpr int est_regs_f16t(int mt, int nt, int kt, int wm, int wn, int mf) {
    return (mt / wm) * (nt / wn) / 64 + 4 * ((mt / wm) / mf) + 4 * ((nt / wn) / mf) +
           2 * ((mt + nt) * kt * 2 / 1024 / (wm * wn)) + 32;
}
constexpr int lds_f16t(int mt, int nt, int kt, int st) { return st * (mt + nt) * kt * 2; }

#define NNJIT_F16T_VARIANT(MT, NT, KT, WM, WN, MF, ST)                                                      \
    {"gemm_f16t_" #MT "x" #NT "x" #KT "_w" #WM "x" #WN "_m" #MF "_s" #ST, FAM_GEMM_F16, MF, (MF == 32 ? 16 : 32), \
     MT, NT, KT, WM, WN, ST, ST - 1, 1, 16, 0, 0, WM * WN * 64, lds_f16t(MT, NT, KT, ST),                     \
     est_regs_f16t(MT, NT, KT, WM, WN, MF), (const void *)&gemm_f16t_kernel<MT, NT, KT, WM, WN, MF, ST>,      \
     &launch_gemm_f16t<MT, NT, KT, WM, WN, MF, ST>, 1, LAYOUT_SWIZZLE, 0}

// The compiled direct-copy configurations (16-byte aligned operands, Nt >= 128).
#define NNJIT_F16T_LIST(X) \
    X(256, 256, 64, 4, 2, 32, 2) \
    X(256, 128, 64, 4, 4, 32, 3) \
    X(256, 256, 64, 2, 4, 32, 2) \
    X(256, 256, 32, 2, 4, 32, 4) \
    X(256, 256, 32, 2, 4, 32, 5) \
    X(256, 256, 32, 4, 2, 32, 4) \
    X(256, 128, 64, 2, 2, 32, 2) \
    X(256, 128, 64, 2, 2, 32, 3) \
    X(256, 128, 64, 4, 2, 32, 2) \
    X(256, 128, 64, 4, 2, 32, 3) \
    X(256, 128, 32, 4, 2, 32, 5) \
    X(128, 256, 64, 2, 2, 32, 2) \
    X(128, 256, 64, 2, 2, 32, 3) \
    X(128, 256, 64, 2, 4, 32, 2) \
    X(128, 256, 64, 2, 4, 32, 3) \
    X(128, 256, 32, 2, 4, 32, 4) \
    X(128, 256, 32, 2, 4, 32, 5) \
    X(128, 128, 64, 2, 2, 32, 2) \
    X(128, 128, 64, 2, 2, 32, 3) \
    X(128, 128, 64, 2, 2, 16, 2) \
    X(128, 128, 64, 2, 2, 16, 3) \
    X(128, 128, 64, 4, 2, 32, 3) \
    X(64, 128, 64, 2, 2, 32, 2) \
    X(64, 128, 64, 2, 2, 32, 3) \
    X(64, 128, 64, 1, 2, 32, 3)

#define NNJIT_F16T_INST(MT, NT, KT, WM, WN, MF, ST) \
    template __global__ void gemm_f16t_kernel<MT, NT, KT, WM, WN, MF, ST>(GemmParams);
NNJIT_F16T_LIST(NNJIT_F16T_INST)

#define NNJIT_F16_INST(MT, NT, WM, WN, MF, ST, PF, VEC) \
    template __global__ void gemm_f16_kernel<MT, NT, WM, WN, MF, ST, PF, VEC>(GemmParams);
NNJIT_F16_LIST(NNJIT_F16_INST)

#if !defined(__HIP_DEVICE_COMPILE__)
#define NNJIT_F16_ENTRY(...) NNJIT_F16_VARIANT(__VA_ARGS__),
#define NNJIT_F16T_ENTRY(...) NNJIT_F16T_VARIANT(__VA_ARGS__),
const Variant kGemmF16Variants[] = {NNJIT_F16_LIST(NNJIT_F16_ENTRY) NNJIT_F16T_LIST(NNJIT_F16T_ENTRY)};
const int kNumGemmF16Variants = sizeof(kGemmF16Variants) / sizeof(kGemmF16Variants[0]);
#endif

}  // namespace nnjit
