// fp32 MatMul / BatchMatMul on the fp32 matrix cores of gfx950.
//
// One workgroup computes an Mt x Nt tile of C for one split of K and one
// batch slice.  This is the paper's tile hierarchy (Fig. 10, Table 1): the
// block tile (x1, y1, r1) = (Nt, Mt, Kt) is staged through LDS (the
// "cache_read" primitive of Table 2), each wave owns a (Mt/WM) x (Nt/WN)
// sub-tile held in accumulator registers (the thread tile; "cache_write": C
// is written once, at the end), and the inner loop over the slab is fully
// unrolled (the "unroll" primitive).  Global loads are 128-bit (heuristic 1).
//
// Matrix-core instructions (operands are per lane of a 64-lane wave):
//   v_mfma_f32_32x32x2_f32:  lane l holds A[i][k], B[k][j] with i = j = l % 32,
//                            k = l / 32; D[i][j] is register 8*(i/8)... see
//                            row_of() below.
//   v_mfma_f32_16x16x4_f32:  i = j = l % 16, k = l / 16.
// Only the pairing of A and B k-slots matters for the product, so lane group
// g takes the K-slab's k in [g*KL, (g+1)*KL) one per instruction; A values
// of a lane are then contiguous in LDS and are read 128 bits at a time.
#include "kcommon.h"

namespace nnjit {

template <int MF> struct Mfma32;
template <> struct Mfma32<32> {
    typedef f32x16 acc_t;
    static constexpr int NR = 16;
    __device__ static __forceinline__ acc_t mma(float a, float b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
    }
    // row of accumulator register r of a lane in lane group g (column = l % 32)
    __device__ static __forceinline__ int row_of(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }
};
template <> struct Mfma32<16> {
    typedef f32x4 acc_t;
    static constexpr int NR = 4;
    __device__ static __forceinline__ acc_t mma(float a, float b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    __device__ static __forceinline__ int row_of(int r, int g) { return 4 * g + r; }
};

// Sliced K: a workgroup holds KS groups of WM x WN waves.  Group g takes the
// K slabs g, g + KS, g + 2 KS, ... of the workgroup's K range through its own
// LDS buffers; at the end the groups' accumulators are added in group order
// through LDS (deterministic).  KS multiplies the waves and the loads in
// flight per CU without a second kernel, which is what small-M products
// (few tiles, long K) need.
template <int MT, int NT, int KT, int WM, int WN, int MF, int ST, int PF, int KS, bool VEC>
__global__ void __launch_bounds__(KS * WM * WN * 64)
gemm_f32_kernel(GemmParams p)
{
    typedef Mfma32<MF> I;
    typedef typename I::acc_t acc_t;
    constexpr int NTG = WM * WN * 64;    // threads of one K group
    constexpr int WTM = MT / WM, WTN = NT / WN;
    constexpr int FM = WTM / MF, FN = WTN / MF;
    // A slab: [Mt][Kt] floats.  Measured on gfx950: a 128-bit LDS read is
    // served 16 lanes (256 bytes) at a time, a 128-bit write 8 lanes (128
    // bytes).  Kt = 16 rows (64 bytes) are unpadded with the 16-byte chunk
    // index XOR-swizzled by (row >> 2) & 3, deeper slabs are padded by 4
    // floats; both keep the 128-bit stores (8 lanes = 128 contiguous bytes)
    // and the fragment reads (16 consecutive rows) free of bank conflicts.
    constexpr bool SWZ = (KT == 16);
    constexpr int SA = SWZ ? KT : KT + 4;
    constexpr int SB = NT + 4;           // B slab: [Kt][Nt + 4] floats
    constexpr int A4 = MT * KT / 4;      // 16-byte chunks of one A slab
    constexpr int B4 = KT * NT / 4;
    constexpr int LA = (A4 + NTG - 1) / NTG;
    constexpr int LB = (B4 + NTG - 1) / NTG;
    constexpr int KG = 64 / MF;          // lane groups along k
    constexpr int KL = KT / KG;          // k values of one lane group per slab
    constexpr int SLAB = MT * SA + KT * SB;                       // floats per buffer
    constexpr int NREG = FM * FN * I::NR;                         // accumulators per lane
    constexpr int LDS_MAIN = KS * ST * SLAB;
    constexpr int LDS_RED = (KS - 1) * NREG * NTG;
    constexpr int LDSF = LDS_MAIN > LDS_RED ? LDS_MAIN : LDS_RED;
    static_assert(FM >= 1 && FN >= 1 && WTM % MF == 0 && WTN % MF == 0, "wave tile");
    static_assert(KL % 4 == 0, "K-slab too small for 128-bit LDS reads");
    static_assert(MT * NT == NTG * NREG, "tile / accumulator count");

    __shared__ __attribute__((aligned(16))) float lds[LDSF];

    const int tid = threadIdx.x;
    const int kgp = tid / NTG, tg = tid % NTG;   // K group, thread within the group
    const int lane = tg & 63, wave = tg >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int li = lane % MF, lg = lane / MF;
    float *gl = lds + kgp * ST * SLAB;            // this group's buffers
    auto As = [&](int buf) { return gl + buf * SLAB; };
    auto Bs = [&](int buf) { return gl + buf * SLAB + MT * SA; };
    auto a_off = [](int row, int chunk) {
        return row * SA + 4 * (SWZ ? (chunk ^ ((row >> 2) & 3)) : chunk);
    };

    // workgroup -> (batch z, split s, tile)
    const int tiles = p.tiles_m * p.tiles_n;
    const int gx = gridDim.x;
    const int logical = xcd_remap(blockIdx.x + gx * blockIdx.z, gx * gridDim.z);
    const int z = logical / gx;
    const int rest = logical - z * gx;
    const int s = rest / tiles;
    const int tile = rest - s * tiles;
    const int tm = tile % p.tiles_m, tn = tile / p.tiles_m;
    const int m0 = tm * MT, n0 = tn * NT;
    const int kbeg = s * p.kchunk;
    const int kend = min(p.K, kbeg + p.kchunk);
    const int nk = kend > kbeg ? (kend - kbeg + KT - 1) / KT : 0;   // slabs of the workgroup
    const int nkg = (nk + KS - 1) / KS;                              // iterations of every group

    const float *A = (const float *)p.A + (long long)z * p.sA;
    const float *B = (const float *)p.B + (long long)z * p.sB;
    float *C = p.C + (long long)z * p.sC;
    const int M = p.M, N = p.N;
    const long long lda = p.lda, ldb = p.ldb;

    // PF slabs are in flight in registers (a ring of PF staging sets), so
    // the loads of slab it+PF are issued while slab it is computed
    f32x4 ra[PF][LA], rb[PF][LB];

    // Loads are branch-free and never followed by value-dependent work: an
    // out-of-range element is read from a zero-filled buffer instead (only
    // the address is selected).  A divergent branch around a load, or a
    // select on its result, would make the compiler wait for every
    // outstanding load before the next slab's loads are issued.
    const float *zero = (const float *)p.zero;
    auto gload = [&](int set, int it) {
        const int k0 = kbeg + (it * KS + kgp) * KT;   // this group's slab of iteration it
#pragma unroll
        for (int l = 0; l < LA; ++l) {
            const int f = tg + l * NTG;
            const int row = f / (KT / 4), c4 = f % (KT / 4);
            const int gm = m0 + row, gk = k0 + c4 * 4;
            const bool okr = (A4 % NTG == 0 || f < A4) && gm < M;
            const float *src = A + (long long)gm * lda + gk;
            f32x4 v;
            if constexpr (VEC) {
                v = *(const f32x4 *)((okr && gk < kend) ? src : zero);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = *((okr && gk + e < kend) ? src + e : zero);
            }
            ra[set][l] = v;
        }
#pragma unroll
        for (int l = 0; l < LB; ++l) {
            const int f = tg + l * NTG;
            const int row = f / (NT / 4), c4 = f % (NT / 4);
            const int gk = k0 + row, gn = n0 + c4 * 4;
            const bool okr = (B4 % NTG == 0 || f < B4) && gk < kend;
            const float *src = B + (long long)gk * ldb + gn;
            f32x4 v;
            if constexpr (VEC) {
                v = *(const f32x4 *)((okr && gn < N) ? src : zero);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = *((okr && gn + e < N) ? src + e : zero);
            }
            rb[set][l] = v;
        }
    };

    auto sstore = [&](int set, int buf) {
        float *as = As(buf), *bs = Bs(buf);
#pragma unroll
        for (int l = 0; l < LA; ++l) {
            const int f = tg + l * NTG;
            if (A4 % NTG == 0 || f < A4) {
                const int row = f / (KT / 4), c4 = f % (KT / 4);
                *(f32x4 *)&as[a_off(row, c4)] = ra[set][l];
            }
        }
#pragma unroll
        for (int l = 0; l < LB; ++l) {
            const int f = tg + l * NTG;
            if (B4 % NTG == 0 || f < B4) {
                const int row = f / (NT / 4), c4 = f % (NT / 4);
                *(f32x4 *)&bs[row * SB + c4 * 4] = rb[set][l];
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
        const float *as = As(buf);
        const float *bs = Bs(buf) + (lg * KL) * SB + wn * WTN + li;
#pragma unroll
        for (int q = 0; q < KL / 4; ++q) {
            f32x4 a[FM];
#pragma unroll
            for (int i = 0; i < FM; ++i)
                a[i] = *(const f32x4 *)&as[a_off(wm * WTM + i * MF + li, lg * (KL / 4) + q)];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                float b[FN];
#pragma unroll
                for (int j = 0; j < FN; ++j) b[j] = bs[(4 * q + e) * SB + j * MF];
#pragma unroll
                for (int i = 0; i < FM; ++i)
#pragma unroll
                    for (int j = 0; j < FN; ++j) acc[i][j] = I::mma(a[i][e], b[j], acc[i][j]);
            }
        }
    };

    // Software pipeline (per K group).  Iteration it's slab is loaded into
    // staging set it % PF at iteration it - PF, stored to LDS buffer it & 1 at
    // iteration it - 1 and multiplied at iteration it.  The loop is unrolled
    // by PF so every set index is a compile-time constant, and its loads and
    // LDS stores are unconditional (slabs past the end read the zero buffer)
    // so the compiler keeps PF slabs in flight; only the matrix-core work is
    // skipped past the end.  Every group runs the same iterations, so the
    // workgroup barriers match.
    if (nk > 0) {
#pragma unroll
        for (int u = 0; u < PF; ++u) gload(u, u);
        if constexpr (ST == 2) {
            sstore(0, 0);
            __syncthreads();
        }
        for (int it0 = 0; it0 < nkg; it0 += PF) {
#pragma unroll
            for (int u = 0; u < PF; ++u) {
                const int it = it0 + u;
                const bool live = it * KS + kgp < nk;
                if constexpr (ST == 2) {
                    gload(u, it + PF);
                    if (live) compute(it & 1);
                    sstore((u + 1) % PF, (it + 1) & 1);
                    __syncthreads();
                } else {
                    __syncthreads();
                    sstore(u, 0);
                    __syncthreads();
                    gload(u, it + PF);
                    if (live) compute(0);
                }
            }
        }
    }

    if constexpr (KS > 1) {
        // groups 1 .. KS-1 hand their accumulators to group 0 through LDS
        __syncthreads();
        if (kgp > 0) {
            float *red = lds + (long long)(kgp - 1) * NREG * NTG;
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int r = 0; r < I::NR; ++r) red[((i * FN + j) * I::NR + r) * NTG + tg] = acc[i][j][r];
        }
        __syncthreads();
        if (kgp > 0) return;
#pragma unroll
        for (int g = 1; g < KS; ++g) {
            const float *red = lds + (long long)(g - 1) * NREG * NTG;
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int r = 0; r < I::NR; ++r) acc[i][j][r] += red[((i * FN + j) * I::NR + r) * NTG + tg];
        }
    }

    const int rbase = m0 + wm * WTM, cbase = n0 + wn * WTN + li;
    // S == 1: C directly; S > 1: this split's partial tile goes to
    // ws[s][z][row][col] and a separate kernel sums the S partials in order
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

template <int MT, int NT, int KT, int WM, int WN, int MF, int ST, int PF, int KS, bool VEC>
static hipError_t launch_gemm_f32(const void *params, dim3 grid, hipStream_t stream)
{
    hipLaunchKernelGGL((gemm_f32_kernel<MT, NT, KT, WM, WN, MF, ST, PF, KS, VEC>), grid, dim3(KS * WM * WN * 64), 0,
                       stream, *(const GemmParams *)params);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// LDS-free ("direct") variant for small M.  Every wave owns a WTM x WTN block
// of C and one K slice; it loads its matrix-core fragments straight from
// global memory (L2-resident operands at these sizes) into a ring of PF
// register sets and never waits at a barrier inside the K loop.  A
// workgroup holds CB column blocks x KS K slices of waves: the CB waves of a
// slice share A rows in L1, and at the end the KS slices of a block are
// added through LDS in slice order (deterministic).  Fragment lane layout as
// above: lane group g takes k in [g*KL, (g+1)*KL) of each K slab, so its A
// values are 16-byte contiguous and its B values are one 4-byte word per k
// (consecutive lanes read consecutive columns, coalesced).
template <int WTM, int WTN, int KT, int CB, int MF, int PF, int KS, bool VEC>
__global__ void __launch_bounds__(CB * KS * 64)
gemm_f32_direct_kernel(GemmParams p)
{
    typedef Mfma32<MF> I;
    typedef typename I::acc_t acc_t;
    constexpr int FM = WTM / MF, FN = WTN / MF;
    constexpr int KG = 64 / MF;          // lane groups along k
    constexpr int KL = KT / KG;          // k values of one lane group per slab
    constexpr int NREG = FM * FN * I::NR;
    static_assert(FM >= 1 && FN >= 1 && KL % 4 == 0, "direct tile");

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int cb = wave % CB, ks = wave / CB;       // column block, K slice
    const int li = lane % MF, lg = lane / MF;

    const int tiles = p.tiles_m * p.tiles_n;
    const int gx = gridDim.x;
    const int logical = xcd_remap(blockIdx.x + gx * blockIdx.z, gx * gridDim.z);
    const int z = logical / gx;
    const int rest = logical - z * gx;
    const int s = rest / tiles;
    const int tile = rest - s * tiles;
    const int tm = tile % p.tiles_m, tn = tile / p.tiles_m;
    const int m0 = tm * WTM, n0 = tn * (CB * WTN) + cb * WTN;
    const int kbeg = s * p.kchunk;
    const int kend = min(p.K, kbeg + p.kchunk);
    const int nk = kend > kbeg ? (kend - kbeg + KT - 1) / KT : 0;
    const int nps = (nk + KS - 1) / KS;              // slabs of one K slice
    const int sl0 = ks * nps;                        // this slice's first slab
    const int nmine = max(0, min(nk - sl0, nps));

    const float *A = (const float *)p.A + (long long)z * p.sA;
    const float *B = (const float *)p.B + (long long)z * p.sB;
    float *C = p.C + (long long)z * p.sC;
    const int M = p.M, N = p.N;
    const long long lda = p.lda, ldb = p.ldb;
    const float *zero = (const float *)p.zero;

    f32x4 ra[PF][FM][KL / 4];
    float rb[PF][FN][KL];
    auto gload = [&](int set, int it) {
        const int k0 = kbeg + (sl0 + it) * KT + lg * KL;
        const bool okk = it < nmine;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int gm = m0 + i * MF + li;
            const float *src = A + (long long)gm * lda + k0;
#pragma unroll
            for (int q = 0; q < KL / 4; ++q) {
                if constexpr (VEC) {
                    ra[set][i][q] = *(const f32x4 *)((okk && gm < M && k0 + 4 * q < kend) ? src + 4 * q : zero);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        ra[set][i][q][e] = *((okk && gm < M && k0 + 4 * q + e < kend) ? src + 4 * q + e : zero);
                }
            }
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int gn = n0 + j * MF + li;
            const float *src = B + (long long)k0 * ldb + gn;
#pragma unroll
            for (int e = 0; e < KL; ++e)
                rb[set][j][e] = *((okk && gn < N && k0 + e < kend) ? src + (long long)e * ldb : zero);
        }
    };

    acc_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < I::NR; ++r) acc[i][j][r] = 0.f;

    auto compute = [&](int set) {
#pragma unroll
        for (int e = 0; e < KL; ++e)
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = I::mma(ra[set][i][e >> 2][e & 3], rb[set][j][e], acc[i][j]);
    };

    // register ring: slab it is loaded PF iterations ahead; loads are
    // unconditional (past the end they read the zero buffer)
#pragma unroll
    for (int u = 0; u < PF; ++u) gload(u, u);
    for (int it0 = 0; it0 < nmine; it0 += PF) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const int it = it0 + u;
            if (it < nmine) compute(u);
            gload(u, it + PF);
        }
    }

    if constexpr (KS > 1) {
        // slices 1 .. KS-1 hand their accumulators to slice 0 through LDS
        __shared__ float red[(KS > 1 ? KS - 1 : 1) * CB * NREG * 64];
        if (ks > 0) {
            float *r = red + ((ks - 1) * CB + cb) * NREG * 64;
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int q = 0; q < I::NR; ++q) r[((i * FN + j) * I::NR + q) * 64 + lane] = acc[i][j][q];
        }
        __syncthreads();
        if (ks > 0) return;
#pragma unroll
        for (int g = 1; g < KS; ++g) {
            const float *r = red + ((g - 1) * CB + cb) * NREG * 64;
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int q = 0; q < I::NR; ++q) acc[i][j][q] += r[((i * FN + j) * I::NR + q) * 64 + lane];
        }
    }

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
                const int row = m0 + i * MF + I::row_of(r, lg), col = n0 + j * MF + li;
                if (row < M && col < N) out[(long long)row * ldo + col] = acc[i][j][r];
            }
}

template <int WTM, int WTN, int KT, int CB, int MF, int PF, int KS, bool VEC>
static hipError_t launch_gemm_f32_direct(const void *params, dim3 grid, hipStream_t stream)
{
    hipLaunchKernelGGL((gemm_f32_direct_kernel<WTM, WTN, KT, CB, MF, PF, KS, VEC>), grid, dim3(CB * KS * 64), 0, stream,
                       *(const GemmParams *)params);
    return hipGetLastError();
}

// Register estimate of the Table 1 formula Reg_thread = x0*r0 + r0*y0 + x0*y0
// for one lane: the accumulator tile (x0*y0 over 64 lanes), the A and B
// fragments of one K step (r0*y0, r0*x0), the global->LDS staging registers,
// and a fixed overhead for addresses and indices.
constexpr int est_regs_f32(int mt, int nt, int kt, int wm, int wn, int mf, int pf) {
    return (mt / wm) * (nt / wn) / 64 + 4 * ((mt / wm) / mf) + ((nt / wn) / mf) +
           pf * ((mt * kt + kt * nt) / (wm * wn * 64)) + 28;
}
constexpr int lds_f32(int mt, int nt, int kt, int st, int ks) {
    return (ks * st * (mt * (kt == 16 ? kt : kt + 4) + kt * (nt + 4)) > (ks - 1) * mt * nt
                ? ks * st * (mt * (kt == 16 ? kt : kt + 4) + kt * (nt + 4))
                : (ks - 1) * mt * nt) * 4;
}

#define NNJIT_F32_VARIANT(MT, NT, KT, WM, WN, MF, ST, PF, KS, VEC)                                        \
    {"gemm_f32_" #MT "x" #NT "x" #KT "_w" #WM "x" #WN "_m" #MF "_s" #ST "_p" #PF "_k" #KS "_v" #VEC,             \
     FAM_GEMM_F32, MF, (MF == 32 ? 2 : 4), MT, NT, KT, WM, WN, ST, PF, KS, (VEC ? 16 : 4), 0, 0,               \
     KS * WM * WN * 64, lds_f32(MT, NT, KT, ST, KS), est_regs_f32(MT, NT, KT, WM, WN, MF, PF),                 \
     (const void *)&gemm_f32_kernel<MT, NT, KT, WM, WN, MF, ST, PF, KS, VEC>,                                 \
     &launch_gemm_f32<MT, NT, KT, WM, WN, MF, ST, PF, KS, VEC>}

// Direct variants: macro tile = WTM x (CB * WTN); waves = CB x KS; no LDS
// staging (only the final K-slice reduction); registers = accumulators +
// PF x (A + B fragments of one slab) + overhead.
constexpr int est_regs_f32d(int wtm, int wtn, int kt, int mf, int pf) {
    return wtm * wtn / 64 + pf * ((wtm / mf) * (kt / (64 / mf)) + (wtn / mf) * (kt / (64 / mf))) + 24;
}
#define NNJIT_F32D_VARIANT(WTM, WTN, KT, CB, MF, PF, KS, VEC)                                                  \
    {"gemm_f32d_" #WTM "x" #WTN "x" #KT "_c" #CB "_m" #MF "_p" #PF "_k" #KS "_v" #VEC, FAM_GEMM_F32, MF,          \
     (MF == 32 ? 2 : 4), WTM, CB * WTN, KT, 1, CB, 0, PF, KS, (VEC ? 16 : 4), 0, 0, CB * KS * 64,                \
     (KS > 1 ? (KS - 1) * CB * WTM * WTN * 4 : 4), est_regs_f32d(WTM, WTN, KT, MF, PF),                         \
     (const void *)&gemm_f32_direct_kernel<WTM, WTN, KT, CB, MF, PF, KS, VEC>,                                   \
     &launch_gemm_f32_direct<WTM, WTN, KT, CB, MF, PF, KS, VEC>}

#define NNJIT_F32D_LIST(X) \
    X(32, 32, 16, 4, 16, 4, 4, true) \
    X(32, 32, 16, 4, 16, 2, 4, true) \
    X(32, 32, 16, 2, 16, 4, 4, true) \
    X(32, 32, 16, 2, 32, 4, 4, true) \
    X(32, 32, 16, 4, 32, 4, 4, true) \
    X(16, 16, 16, 4, 16, 4, 4, true) \
    X(16, 16, 16, 4, 16, 8, 4, true) \
    X(32, 16, 16, 4, 16, 4, 4, true) \
    X(16, 32, 16, 4, 16, 4, 4, true) \
    X(32, 64, 16, 2, 32, 4, 4, true) \
    X(64, 32, 16, 2, 32, 4, 4, true) \
    X(32, 32, 32, 4, 16, 2, 4, true) \
    X(32, 32, 32, 2, 32, 2, 4, true)

#define NNJIT_F32D_INST(WTM, WTN, KT, CB, MF, PF, KS, VEC) \
    template __global__ void gemm_f32_direct_kernel<WTM, WTN, KT, CB, MF, PF, KS, VEC>(GemmParams);
NNJIT_F32D_LIST(NNJIT_F32D_INST)

// The compiled fp32 configurations (the family's full set; the lite space of
// a shape is a pruned, ordered subset).  Tile edges are powers of two
// (heuristic 2).  The last entries load element by element, for operands
// that are not 16-byte aligned.
#define NNJIT_F32_LIST(X) \
    X(64, 64, 16, 2, 2, 32, 2, 2, 2, true) \
    X(64, 64, 16, 2, 2, 32, 2, 2, 4, true) \
    X(64, 32, 16, 2, 2, 16, 2, 4, 4, true) \
    X(32, 64, 16, 2, 2, 16, 2, 4, 4, true) \
    X(64, 64, 16, 2, 2, 16, 2, 4, 4, true) \
    X(32, 32, 16, 2, 2, 16, 2, 4, 4, true) \
    X(64, 32, 32, 2, 2, 16, 2, 2, 4, true) \
    X(32, 64, 32, 2, 2, 16, 2, 2, 4, true) \
    X(64, 64, 32, 2, 2, 16, 2, 2, 4, true) \
    X(64, 32, 16, 2, 1, 32, 2, 4, 4, true) \
    X(32, 64, 16, 1, 2, 32, 2, 4, 4, true) \
    X(64, 64, 32, 2, 2, 32, 2, 2, 2, true) \
    X(64, 64, 16, 2, 2, 16, 2, 2, 2, true) \
    X(64, 64, 16, 2, 2, 16, 2, 2, 4, true) \
    X(64, 32, 16, 2, 2, 16, 2, 2, 2, true) \
    X(64, 32, 16, 2, 2, 16, 2, 2, 4, true) \
    X(32, 64, 16, 2, 2, 16, 2, 2, 2, true) \
    X(32, 64, 16, 2, 2, 16, 2, 2, 4, true) \
    X(32, 32, 16, 2, 2, 16, 2, 2, 4, true) \
    X(64, 32, 32, 2, 1, 32, 2, 2, 4, true) \
    X(32, 64, 32, 1, 2, 32, 2, 2, 4, true) \
    X(128, 64, 16, 2, 2, 32, 2, 2, 2, true) \
    X(64, 128, 16, 2, 2, 32, 2, 2, 2, true) \
    X(128, 128, 16, 2, 2, 32, 2, 1, 2, true) \
    X(256, 128, 16, 2, 2, 32, 2, 1, 1, true) \
    X(128, 256, 16, 2, 2, 32, 2, 1, 1, true) \
    X(256, 256, 16, 2, 2, 32, 2, 1, 1, true) \
    X(256, 128, 16, 4, 2, 32, 2, 1, 1, true) \
    X(256, 128, 16, 4, 2, 32, 2, 2, 1, true) \
    X(128, 128, 16, 2, 2, 32, 2, 1, 1, true) \
    X(128, 128, 16, 2, 2, 32, 2, 2, 1, true) \
    X(128, 128, 32, 2, 2, 32, 2, 1, 1, true) \
    X(128, 128, 16, 2, 2, 32, 1, 1, 1, true) \
    X(128, 128, 16, 1, 2, 32, 2, 1, 1, true) \
    X(128, 64, 16, 2, 2, 32, 2, 1, 1, true) \
    X(128, 64, 16, 2, 2, 32, 2, 2, 1, true) \
    X(128, 64, 32, 2, 2, 32, 2, 2, 1, true) \
    X(64, 128, 16, 2, 2, 32, 2, 1, 1, true) \
    X(64, 128, 16, 2, 2, 32, 2, 2, 1, true) \
    X(64, 128, 32, 2, 2, 32, 2, 2, 1, true) \
    X(64, 64, 16, 2, 2, 32, 2, 1, 1, true) \
    X(64, 64, 16, 2, 2, 32, 2, 2, 1, true) \
    X(64, 64, 16, 2, 2, 32, 2, 4, 1, true) \
    X(64, 64, 32, 2, 2, 32, 2, 2, 1, true) \
    X(64, 64, 64, 2, 2, 32, 2, 1, 1, true) \
    X(64, 64, 64, 2, 2, 32, 2, 2, 1, true) \
    X(64, 64, 64, 2, 2, 16, 2, 2, 1, true) \
    X(128, 64, 64, 2, 2, 32, 2, 2, 1, true) \
    X(64, 128, 64, 2, 2, 32, 2, 2, 1, true) \
    X(32, 64, 64, 1, 2, 32, 2, 2, 1, true) \
    X(64, 32, 64, 2, 1, 32, 2, 2, 1, true) \
    X(32, 64, 64, 2, 2, 16, 2, 2, 1, true) \
    X(64, 32, 64, 2, 2, 16, 2, 2, 1, true) \
    X(32, 32, 64, 2, 2, 16, 2, 2, 1, true) \
    X(32, 32, 64, 1, 1, 32, 2, 2, 1, true) \
    X(64, 64, 16, 2, 2, 16, 2, 2, 1, true) \
    X(64, 64, 16, 2, 2, 32, 1, 1, 1, true) \
    X(64, 64, 16, 2, 2, 32, 1, 2, 1, true) \
    X(64, 64, 16, 1, 1, 32, 2, 2, 1, true) \
    X(32, 64, 16, 1, 2, 32, 2, 2, 1, true) \
    X(32, 64, 32, 1, 2, 32, 2, 2, 1, true) \
    X(64, 32, 16, 2, 1, 32, 2, 2, 1, true) \
    X(64, 32, 32, 2, 1, 32, 2, 2, 1, true) \
    X(32, 32, 16, 1, 1, 32, 2, 2, 1, true) \
    X(32, 32, 32, 1, 1, 32, 2, 2, 1, true) \
    X(32, 32, 16, 2, 2, 16, 2, 1, 1, true) \
    X(32, 32, 16, 2, 2, 16, 2, 2, 1, true) \
    X(32, 32, 16, 2, 2, 16, 2, 4, 1, true) \
    X(32, 64, 16, 2, 2, 16, 2, 2, 1, true) \
    X(32, 64, 16, 2, 2, 16, 2, 4, 1, true) \
    X(64, 32, 16, 2, 2, 16, 2, 2, 1, true) \
    X(64, 32, 16, 2, 2, 16, 2, 4, 1, true) \
    X(16, 64, 16, 1, 2, 16, 2, 2, 1, true) \
    X(16, 64, 32, 1, 4, 16, 2, 2, 1, true) \
    X(64, 64, 16, 2, 2, 32, 2, 1, 1, false) \
    X(32, 32, 16, 1, 1, 32, 2, 1, 1, false)

#define NNJIT_F32_INST(MT, NT, KT, WM, WN, MF, ST, PF, KS, VEC) \
    template __global__ void gemm_f32_kernel<MT, NT, KT, WM, WN, MF, ST, PF, KS, VEC>(GemmParams);
NNJIT_F32_LIST(NNJIT_F32_INST)

#if !defined(__HIP_DEVICE_COMPILE__)
#define NNJIT_F32_ENTRY(...) NNJIT_F32_VARIANT(__VA_ARGS__),
#define NNJIT_F32D_ENTRY(...) NNJIT_F32D_VARIANT(__VA_ARGS__),
const Variant kGemmF32Variants[] = {NNJIT_F32_LIST(NNJIT_F32_ENTRY) NNJIT_F32D_LIST(NNJIT_F32D_ENTRY)};
const int kNumGemmF32Variants = sizeof(kGemmF32Variants) / sizeof(kGemmF32Variants[0]);
#endif

}  // namespace nnjit
