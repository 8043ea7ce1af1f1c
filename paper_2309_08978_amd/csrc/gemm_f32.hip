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
//
// LAY (A slab layout) and ROLL (K steps of a slab as a loop) exist so that
// the offline primitive benchmark can compare settings one at a time; the
// default layout is the swizzle for 16-deep slabs and padding otherwise,
// and the default is fully unrolled.
template <int MT, int NT, int KT, int WM, int WN, int MF, int ST, int PF, int KS, bool VEC,
          int LAY = (KT == 16 ? LAYOUT_SWIZZLE : LAYOUT_PAD), bool ROLL = false>
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
    constexpr bool SWZ = (LAY == LAYOUT_SWIZZLE);
    constexpr int SA = (LAY == LAYOUT_PAD) ? KT + 4 : KT;
    static_assert(!SWZ || KT % 16 == 0, "the swizzle permutes groups of four 16-byte chunks");
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
    int tm, tn;
    tile_of(tile, p.tiles_m, p.tiles_n, p.group_m, tm, tn);
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
        auto step = [&](int q) {
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
        };
        if constexpr (ROLL) {
#pragma unroll 1
            for (int q = 0; q < KL / 4; ++q) step(q);
        } else {
#pragma unroll
            for (int q = 0; q < KL / 4; ++q) step(q);
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

template <int MT, int NT, int KT, int WM, int WN, int MF, int ST, int PF, int KS, bool VEC,
          int LAY = (KT == 16 ? LAYOUT_SWIZZLE : LAYOUT_PAD), bool ROLL = false>
static hipError_t launch_gemm_f32(const void *params, dim3 grid, hipStream_t stream)
{
    hipLaunchKernelGGL((gemm_f32_kernel<MT, NT, KT, WM, WN, MF, ST, PF, KS, VEC, LAY, ROLL>), grid,
                       dim3(KS * WM * WN * 64), 0, stream, *(const GemmParams *)params);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Wave-private K slices ("gemm_f32w") for small-M products.  A workgroup of
// KS waves computes one Mt x Nt tile; wave w takes the K slabs w, w + KS,
// w + 2 KS, ... of the workgroup's K range into its own LDS region with
// global_load_lds_dwordx4 (ST stages) and multiplies them with no barrier in
// the K loop: it waits only for its own copies, by count.  At the end the KS
// partial tiles are added through LDS in wave order (deterministic), each
// wave summing and storing its share of the tile.  Against the shared-slab
// kernel above this gives up operand sharing between waves for a deeper
// pipeline (ST - 1 slabs per wave in flight) and no workgroup lock-step.
//
// Layouts (Kt = 16): A slab [Mt rows][16 floats], the 16-byte piece p of row
// r at piece p ^ ((r >> 2) & 3), so 16 consecutive rows read at one piece hit
// distinct banks; B slab [16 k rows][Nt floats] in 1 KiB copy chunks of R
// rows, each chunk followed by a 16 R-byte gap, so that rows k and k + 8,
// which the two half-waves read in the same instruction, sit on opposite
// halves of the 64 banks.  Lane group g (l / 32) takes k in [8g, 8g + 8) of
// a slab, as in the kernel above.
template <int MT, int NT, int KS, int ST>
__global__ void __launch_bounds__(KS * 64)
gemm_f32w_kernel(GemmParams p)
{
    typedef Mfma32<32> I;
    typedef typename I::acc_t acc_t;
    constexpr int KT = 16;
    constexpr int FM = MT / 32, FN = NT / 32;
    constexpr int A_BYTES = MT * KT * 4;
    constexpr int B_ROW = NT * 4;
    constexpr int RB = 1024 / B_ROW;               // B rows per copy chunk
    constexpr int B_CHUNK = 1024 + 16 * RB;        // chunk plus its bank-half gap
    constexpr int NBC = KT / RB;                   // B copies per slab
    constexpr int NA = A_BYTES / 1024;             // A copies per slab
    constexpr int NCOPY = NA + NBC;
    constexpr int STAGE = A_BYTES + NBC * B_CHUNK;
    constexpr int WAVE_LDS = ST * STAGE;
    constexpr int NREG = FM * FN * I::NR;
    constexpr int RED = KS * NREG * 64 * 4;
    constexpr int LDS_BYTES = KS * WAVE_LDS > RED ? KS * WAVE_LDS : RED;
    static_assert(MT % 32 == 0 && NT % 32 == 0 && NT <= 256 && A_BYTES % 1024 == 0, "tile");
    static_assert(NREG % KS == 0, "epilogue share");
    static_assert((ST - 2) * NCOPY <= 63, "copies in flight exceed the vmcnt range");

    __shared__ __attribute__((aligned(1024))) char smem[LDS_BYTES];
    typedef __attribute__((address_space(3))) char lds_char;

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const int li = lane & 31, lg = lane >> 5;

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
    const int nmine = nk > wave_u ? (nk - wave_u + KS - 1) / KS : 0;    // slabs of this wave

    const float *A = (const float *)p.A + (long long)z * p.sA;
    const float *B = (const float *)p.B + (long long)z * p.sB;
    float *C = p.C + (long long)z * p.sC;
    const int M = p.M, N = p.N;
    const long long lda = p.lda, ldb = p.ldb;
    const float *zero = (const float *)p.zero;
    lds_char *mine = (lds_char *)smem + wave_u * WAVE_LDS;

    // per-lane copy sources for slab 0 of the workgroup's range
    const float *a_src[NA];
    int a_k[NA];
    bool a_ok[NA];
#pragma unroll
    for (int c = 0; c < NA; ++c) {
        const int row = 16 * c + (lane >> 2);
        const int piece = (lane & 3) ^ ((row >> 2) & 3);
        a_ok[c] = m0 + row < M;
        a_k[c] = kbeg + 4 * piece;
        a_src[c] = A + (long long)(a_ok[c] ? m0 + row : 0) * lda + kbeg + 4 * piece;
    }
    const float *b_src[NBC];
    int b_k[NBC];
    bool b_ok[NBC];
#pragma unroll
    for (int c = 0; c < NBC; ++c) {
        const int row = RB * c + lane / (NT / 4);
        const int col = 4 * (lane % (NT / 4));
        b_ok[c] = n0 + col < N;
        b_k[c] = kbeg + row;
        b_src[c] = B + (long long)(kbeg + row) * ldb + (b_ok[c] ? n0 + col : 0);
    }

    // copy this wave's kk-th slab into stage st (past the wave's last slab the
    // sources are the zero buffer, so every wave issues the same copies)
    auto copy_slab = [&](int st, int kk) {
        const int sl = wave_u + kk * KS;
        const bool live = sl < nk;
        const int dk = sl * KT;
        const long long db = (long long)dk * ldb;
        lds_char *dst = mine + st * STAGE;
#pragma unroll
        for (int c = 0; c < NA; ++c) {
            const bool ok = live && a_ok[c] && a_k[c] + dk < kend;
            copy16_to_lds(ok ? a_src[c] + dk : zero, (unsigned)(uintptr_t)(dst + 1024 * c));
        }
#pragma unroll
        for (int c = 0; c < NBC; ++c) {
            const bool ok = live && b_ok[c] && b_k[c] + dk < kend;
            copy16_to_lds(ok ? b_src[c] + db : zero, (unsigned)(uintptr_t)(dst + A_BYTES + B_CHUNK * c));
        }
    };
    // the same copies for a slab that lies wholly inside [kbeg, kend): no
    // checks (rows past M and columns past N were pointed at row / column 0
    // above; what they bring reaches only outputs that are never stored)
    auto copy_full = [&](int st, int kk) {
        const int dk = (wave_u + kk * KS) * KT;
        const long long db = (long long)dk * ldb;
        lds_char *dst = mine + st * STAGE;
#pragma unroll
        for (int c = 0; c < NA; ++c) copy16_to_lds(a_src[c] + dk, (unsigned)(uintptr_t)(dst + 1024 * c));
#pragma unroll
        for (int c = 0; c < NBC; ++c)
            copy16_to_lds(b_src[c] + db, (unsigned)(uintptr_t)(dst + A_BYTES + B_CHUNK * c));
    };
    const int nfull = kend > kbeg ? (kend - kbeg) / KT : 0;                    // whole slabs of the range
    const int nfull_mine = nfull > wave_u ? (nfull - wave_u + KS - 1) / KS : 0;  // ... of this wave

    acc_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < I::NR; ++r) acc[i][j][r] = 0.f;

    // fragments of one slab: FM A rows of 8 k, 8 k rows of FN B columns
    auto read_frags = [&](int st, f32x8 (&a)[FM], float (&b)[8][FN]) {
        lds_char *sa = mine + st * STAGE;
        lds_char *sb = sa + A_BYTES;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int row = 32 * i + li;
            const int sw = (row >> 2) & 3;
            const f32x4 lo = *(__attribute__((address_space(3))) f32x4 *)(sa + row * 64 + 16 * ((2 * lg) ^ sw));
            const f32x4 hi = *(__attribute__((address_space(3))) f32x4 *)(sa + row * 64 + 16 * ((2 * lg + 1) ^ sw));
            a[i] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        }
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int k = 8 * lg + t;
            lds_char *brow = sb + (k / RB) * B_CHUNK + (k % RB) * B_ROW;
#pragma unroll
            for (int j = 0; j < FN; ++j) b[t][j] = *(__attribute__((address_space(3))) float *)(brow + 4 * (32 * j + li));
        }
    };
    auto mma_slab = [&](const f32x8 (&a)[FM], const float (&b)[8][FN]) {
#pragma unroll
        for (int t = 0; t < 8; ++t)
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = I::mma(a[i][t], b[t][j], acc[i][j]);
    };

    // one slab: every fragment read is issued before the first MFMA (the
    // reads return in order, so MFMA t waits only for the reads it uses and
    // the LDS latency is paid once per slab rather than once per step)
    auto compute = [&](int st) {
        f32x8 a[FM];
        float b[8][FN];
        read_frags(st, a, b);
        mma_slab(a, b);
        __builtin_amdgcn_sched_group_barrier(0x100, FM * 2 + 8 * FN, 0);   // all LDS reads first
        __builtin_amdgcn_sched_group_barrier(0x008, 8 * FM * FN, 0);       // then the MFMAs
    };

#pragma unroll
    for (int u = 0; u < ST - 1; ++u) copy_slab(u, u);
    // ST iterations at a time.  While every slab copied in a group is whole
    // (and so is every slab multiplied), the group is one branch-free block:
    // unchecked copies that the scheduler can place among the MFMAs.  The
    // rest runs with checked copies and a guard per slab.  Both issue NCOPY
    // copies per iteration, so the counted waits are the same.
    int it0 = 0;
    if constexpr (ST >= 4 && FM * FN >= 2) {
        static_assert(ST % 2 == 0, "the two register sets alternate within a group of ST slabs");
        // with four or more stages and at least two accumulator tiles (a
        // slab of >= 16 MFMAs, long enough to cover a copy with one fewer
        // slab in flight) the group also reads slab it + 1 into a second
        // register set while the MFMAs of slab it run (the reads interleaved
        // with them), keeping ST - 3 slabs' copies in flight
        if (2 * ST - 1 <= nfull_mine) {
            f32x8 fa[2][FM];
            float fb[2][8][FN];
            wait_vmcnt<(ST - 2) * NCOPY>();   // slab 0
            read_frags(0, fa[0], fb[0]);
            for (; it0 + 2 * ST - 1 <= nfull_mine; it0 += ST) {
#pragma unroll
                for (int u = 0; u < ST; ++u) {
                    // slab it0 + u + 1 has landed once at most the ST - 3
                    // slabs after it are pending; this wave's reads of the
                    // stage about to be refilled (slab it0 + u - 1) are done
                    wait_vmcnt<(ST - 3) * NCOPY>();
                    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
                    copy_full((u + ST - 1) % ST, it0 + u + ST - 1);
                    read_frags((u + 1) % ST, fa[(u + 1) & 1], fb[(u + 1) & 1]);
                    mma_slab(fa[u & 1], fb[u & 1]);
#pragma unroll
                    for (int q = 0; q < 8 * FM * FN; ++q) {
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
                        if (q < FM * 2 + 8 * FN) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
                    }
                }
            }
            // the reads of slab it0 issued by the last group are not used: the
            // loop below reads every slab it multiplies itself
        }
    } else {
        for (; it0 + 2 * ST - 1 <= nfull_mine; it0 += ST) {
#pragma unroll
            for (int u = 0; u < ST; ++u) {
                // slab it0 + u has landed once at most the ST - 2 later
                // slabs' copies are pending; this wave's reads of the stage
                // about to be refilled (multiplied in the previous iteration)
                // are complete
                wait_vmcnt<(ST - 2) * NCOPY>();
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
                copy_full((u + ST - 1) % ST, it0 + u + ST - 1);
                compute(u);
            }
        }
    }
    for (; it0 < nmine; it0 += ST) {
#pragma unroll
        for (int u = 0; u < ST; ++u) {
            const int it = it0 + u;
            wait_vmcnt<(ST - 2) * NCOPY>();
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            copy_slab((u + ST - 1) % ST, it + ST - 1);
            if (it < nmine) compute(u);
        }
    }
    wait_vmcnt<0>();   // no copy may still target LDS when the region is reused
    __syncthreads();

    // every wave's partial tile to LDS, then wave w adds register slots
    // [w NREG / KS, (w + 1) NREG / KS) of all KS partials in wave order
    float *out = C;
    long long ldo = p.ldc;
    if (p.S > 1) {
        out = p.ws + ((long long)s * p.batch + z) * (long long)M * N;
        ldo = N;
    }
    constexpr int SHARE = NREG / KS;
    auto store_slot = [&](int e, float v) {
        const int i = e / (FN * I::NR), j = (e / I::NR) % FN, r = e % I::NR;
        const int row = m0 + 32 * i + I::row_of(r, lg), col = n0 + 32 * j + li;
        if (row < M && col < N) out[(long long)row * ldo + col] = v;
    };
    if constexpr (SHARE % 4 == 0) {
        // four consecutive slots per lane and 16-byte LDS accesses:
        // quad q of wave w at red4[(w NREG / 4 + q) 64 + lane]
        typedef __attribute__((address_space(3))) f32x4 lds_f32x4;
        lds_f32x4 *red4 = (lds_f32x4 *)smem;
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int r4 = 0; r4 < I::NR / 4; ++r4) {
                    const f32x4 v = {acc[i][j][4 * r4], acc[i][j][4 * r4 + 1], acc[i][j][4 * r4 + 2], acc[i][j][4 * r4 + 3]};
                    red4[(wave * (NREG / 4) + (i * FN + j) * (I::NR / 4) + r4) * 64 + lane] = v;
                }
        __syncthreads();
#pragma unroll
        for (int qq = 0; qq < SHARE / 4; ++qq) {
            const int e0 = wave * SHARE + 4 * qq;
            f32x4 v = red4[(e0 / 4) * 64 + lane];
#pragma unroll
            for (int w = 1; w < KS; ++w) v += red4[(w * (NREG / 4) + e0 / 4) * 64 + lane];
#pragma unroll
            for (int c = 0; c < 4; ++c) store_slot(e0 + c, v[c]);
        }
    } else {
        float *red = (float *)smem;
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int r = 0; r < I::NR; ++r) red[((wave * NREG) + (i * FN + j) * I::NR + r) * 64 + lane] = acc[i][j][r];
        __syncthreads();
#pragma unroll
        for (int q = 0; q < SHARE; ++q) {
            const int e = wave * SHARE + q;              // register slot (i, j, r)
            float v = red[e * 64 + lane];
#pragma unroll
            for (int w = 1; w < KS; ++w) v += red[(w * NREG + e) * 64 + lane];
            store_slot(e, v);
        }
    }
}

template <int MT, int NT, int KS, int ST>
static hipError_t launch_gemm_f32w(const void *params, dim3 grid, hipStream_t stream)
{
    hipLaunchKernelGGL((gemm_f32w_kernel<MT, NT, KS, ST>), grid, dim3(KS * 64), 0, stream, *(const GemmParams *)params);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Shared-slab direct-copy variant ("gemm_f32t") for large products: the
// workgroup's waves share one A slab and one B slab per stage, as in
// gemm_f32_kernel, but the slabs go global -> LDS by global_load_lds_dwordx4
// (no staging registers, no LDS store instructions) and are waited for by
// count, with ST stages and one barrier per slab (the register-staged kernel's
// __syncthreads() drains every load in flight at each slab).
//
// Layouts (Kt = 16): A slab [Mt rows][16 floats] with the 16-byte piece p of
// row r at slot p ^ ((r >> 2) & 3) (as in gemm_f32w); B slab [16 k rows][Nt
// floats] with the 16-byte piece p of row k at slot p ^ (8 ((k >> 3) & 1)):
// rows k and k + 8, which the two half-waves read in one ds_read_b32, then
// sit on opposite halves of the 64 banks.  A copy writes 1 KiB contiguously
// at a wave-uniform LDS base (lane l at base + 16 l), so both swizzles are
// made by choosing which global piece each lane fetches.
template <int MT, int NT, int WM, int WN, int ST, bool SK = false>
__global__ void __launch_bounds__(WM * WN * 64)
gemm_f32t_kernel(GemmParams p)
{
    typedef Mfma32<32> I;
    typedef typename I::acc_t acc_t;
    constexpr int KT = 16;
    constexpr int NW = WM * WN;
    constexpr int WTM = MT / WM, WTN = NT / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    constexpr int A_BYTES = MT * KT * 4;
    constexpr int B_ROW = NT * 4;
    constexpr int B_BYTES = KT * B_ROW;
    constexpr int STAGE = A_BYTES + B_BYTES;
    constexpr int LA = A_BYTES / 1024 / NW, LB = B_BYTES / 1024 / NW;   // copies per wave and slab
    constexpr int LC = LA + LB;
    static_assert(LA * NW * 1024 == A_BYTES && LB * NW * 1024 == B_BYTES, "copies must split evenly over waves");
    static_assert(NT >= 64 && (NT & (NT - 1)) == 0, "B rows of a power of two >= 256 bytes");
    static_assert(FM >= 1 && FN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "wave tile");
    static_assert(ST >= 2 && (ST - 2) * LC <= 63, "copies in flight exceed the vmcnt range");

    __shared__ __attribute__((aligned(1024))) char smem[ST * STAGE];
    typedef __attribute__((address_space(3))) char lds_char;

    const int tiles = p.tiles_m * p.tiles_n;
    const int gx = gridDim.x;
    const int logical = xcd_remap(blockIdx.x + gx * blockIdx.z, gx * gridDim.z);
    const int M = p.M, N = p.N;
    const long long lda = p.lda, ldb = p.ldb;
    const float *zero = (const float *)p.zero;
    auto stage_base = [&](int u) -> lds_char * { return (lds_char *)smem + u * STAGE; };

    // The workgroup's pieces of work: one (tile, split) in the tiled mode;
    // consecutive (tile, K-slab range) segments of its share of units in the
    // stream-K mode (at most one tile is begun and one ended mid-K).
    long long su = 0, su_end = 1;
    if constexpr (SK) {
        su = (long long)logical * p.units / p.sk_wgs;
        su_end = (long long)(logical + 1) * p.units / p.sk_wgs;
    }
    for (bool first = true; su < su_end; first = false) {
    int z, s, tile, kbeg, kend;
    bool partial = false;
    if constexpr (SK) {
        z = 0;
        s = 0;
        tile = (int)(su / p.nslab);
        const int ks = (int)(su - (long long)tile * p.nslab);
        const int ke = (int)min((long long)p.nslab, ks + (su_end - su));
        kbeg = ks * KT;
        kend = min(p.K, ke * KT);
        partial = ks > 0 || ke < p.nslab;
        su += ke - ks;
    } else {
        z = logical / gx;
        const int rest = logical - z * gx;
        s = rest / tiles;
        tile = rest - s * tiles;
        kbeg = s * p.kchunk;
        kend = min(p.K, kbeg + p.kchunk);
        su = su_end;
    }
    int tm, tn;
    tile_of(tile, p.tiles_m, p.tiles_n, p.group_m, tm, tn);
    const int m0 = tm * MT, n0 = tn * NT;
    const int nk = kend > kbeg ? (kend - kbeg + KT - 1) / KT : 0;
    const float *A = (const float *)p.A + (long long)z * p.sA;
    const float *B = (const float *)p.B + (long long)z * p.sB;
    float *C = p.C + (long long)z * p.sC;
    // the LDS stages are reused: every wave must be done reading the previous
    // segment's slabs before this one's copies land
    if (SK && !first) lds_barrier();
    // The lane's indices are taken afresh in every segment through an opaque
    // copy of the thread id: the lane-dependent addresses derived from them
    // are then computed per segment instead of being held in registers
    // across the segment loop.
    int tid = threadIdx.x;
    if constexpr (SK) asm volatile("v_mov_b32 %0, %0" : "+v"(tid));
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const int li = lane & 31, lg = lane >> 5;

    // per-lane sources of this wave's copies for the split's first slab; copy
    // j of the wave fills 1 KiB chunk c = wave + j NW of the A or B slab
    const float *a_src[LA];
    int a_k[LA];
    bool a_ok[LA];
#pragma unroll
    for (int j = 0; j < LA; ++j) {
        const int row = 16 * (wave + j * NW) + (lane >> 2);
        const int piece = (lane & 3) ^ ((row >> 2) & 3);
        a_ok[j] = m0 + row < M;
        a_k[j] = kbeg + 4 * piece;
        a_src[j] = A + (long long)(a_ok[j] ? m0 + row : 0) * lda + kbeg + 4 * piece;
    }
    const float *b_src[LB];
    int b_k[LB];
    bool b_ok[LB];
#pragma unroll
    for (int j = 0; j < LB; ++j) {
        const int o = 1024 * (wave + j * NW) + 16 * lane;
        const int k = o / B_ROW, slot = (o % B_ROW) >> 4;
        const int col = 4 * (slot ^ (((k >> 3) & 1) << 3));
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

    // fragments of one slab: lane group g takes k in [8g, 8g + 8)
    auto read_frags = [&](int stage, f32x8 (&a)[FM], float (&b)[8][FN]) {
        lds_char *sa = stage_base(stage);
        lds_char *sb = sa + A_BYTES;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int row = wm * WTM + 32 * i + li;
            const int sw = (row >> 2) & 3;
            const f32x4 lo = *(__attribute__((address_space(3))) f32x4 *)(sa + row * 64 + 16 * ((2 * lg) ^ sw));
            const f32x4 hi = *(__attribute__((address_space(3))) f32x4 *)(sa + row * 64 + 16 * ((2 * lg + 1) ^ sw));
            a[i] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        }
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            lds_char *brow = sb + (8 * lg + t) * B_ROW;
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int cc = wn * WTN + 32 * j + li;
                b[t][j] = *(__attribute__((address_space(3))) float *)(brow + 16 * ((cc >> 2) ^ (lg << 3)) + 4 * (cc & 3));
            }
        }
    };
    auto mma_slab = [&](const f32x8 (&a)[FM], const float (&b)[8][FN]) {
#pragma unroll
        for (int t = 0; t < 8; ++t)
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = I::mma(a[i][t], b[t][j], acc[i][j]);
    };

    // one slab: every fragment read is issued before the first MFMA
    auto compute = [&](int stage) {
        f32x8 a[FM];
        float b[8][FN];
        read_frags(stage, a, b);
        mma_slab(a, b);
        __builtin_amdgcn_sched_group_barrier(0x100, FM * 2 + 8 * FN, 0);   // all LDS reads first
        __builtin_amdgcn_sched_group_barrier(0x008, 8 * FM * FN, 0);       // then the MFMAs
    };

    // slab kk is copied into stage kk % ST while slab kk - ST + 1 is
    // multiplied; one barrier per slab
#pragma unroll
    for (int u = 0; u < ST - 1; ++u) copy_slab(u, u);
    // ST slabs at a time.  While every slab copied in a group is whole (and
    // so is every slab multiplied), the group is one branch-free block with
    // unchecked copies that the scheduler can place among the MFMAs; the
    // rest runs with checked copies and a guard per slab.  Both issue the
    // same copies per slab, so the counted waits are the same.
    int it0 = 0;
    if constexpr (ST == 4) {
        // four stages: the main part runs one slab ahead -- the wait and
        // barrier at iteration it make slab it + 1 visible, and its fragments
        // are read into the other register set while slab it's MFMAs run
        // (one slab fewer of copies in flight)
        if (2 * ST - 1 <= nfull) {
            f32x8 fa[2][FM];
            float fb[2][8][FN];
            wait_vmcnt<(ST - 2) * LC>();   // slab 0
            lds_barrier();
            read_frags(0, fa[0], fb[0]);
            for (; it0 + 2 * ST - 1 <= nfull; it0 += ST) {
#pragma unroll
                for (int u = 0; u < ST; ++u) {
                    // this wave's copies of slab it0 + u + 1 are done once at
                    // most the copies of the ST - 3 slabs after it are
                    // pending; the barrier makes every wave's copies visible
                    // and frees the stage of slab it0 + u - 1, whose reads
                    // were issued in the two previous iterations
                    wait_vmcnt<(ST - 3) * LC>();
                    lds_barrier();
                    copy_full((u + ST - 1) % ST, it0 + u + ST - 1);
                    read_frags((u + 1) % ST, fa[(u + 1) & 1], fb[(u + 1) & 1]);
                    mma_slab(fa[u & 1], fb[u & 1]);
#pragma unroll
                    for (int q = 0; q < 8 * FM * FN; ++q) {
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
                        if (q < FM * 2 + 8 * FN) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
                    }
                }
            }
            // the fragments of slab it0 read by the last iteration go unused:
            // the loop below reads every slab it multiplies itself
        }
    } else {
        for (; it0 + 2 * ST - 1 <= nfull; it0 += ST) {
#pragma unroll
            for (int u = 0; u < ST; ++u) {
                // this wave's copies of slab it0 + u are done once at most the copies
                // of the ST - 2 later slabs are pending; the barrier then makes
                // every wave's copies visible and frees the stage multiplied in
                // the previous iteration
                wait_vmcnt<(ST - 2) * LC>();
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
            wait_vmcnt<(ST - 2) * LC>();
            lds_barrier();
            copy_slab((u + ST - 1) % ST, it + ST - 1);
            if (it < nk) compute(u);
        }
    }
    wait_vmcnt<0>();   // no copy may still target LDS when the workgroup (or segment) ends

    const int rbase = m0 + wm * WTM, cbase = n0 + wn * WTN + li;
    if (SK && partial) {
        // a piece of a tile several workgroups share: the whole Mt x Nt
        // partial tile to this workgroup's slot (first piece 2w, last 2w + 1)
        float *slot = p.ws + (long long)(2 * logical + (first ? 0 : 1)) * (MT * NT);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int r = 0; r < I::NR; ++r) {
                    const int row = wm * WTM + 32 * i + I::row_of(r, lg), col = wn * WTN + li + 32 * j;
                    slot[row * NT + col] = acc[i][j][r];
                }
    } else {
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
                    const int row = rbase + 32 * i + I::row_of(r, lg), col = cbase + 32 * j;
                    if (row < M && col < N) out[(long long)row * ldo + col] = acc[i][j][r];
                }
    }
    }   // segments
}

template <int MT, int NT, int WM, int WN, int ST>
static hipError_t launch_gemm_f32t(const void *params, dim3 grid, hipStream_t stream)
{
    const GemmParams &p = *(const GemmParams *)params;
    if (p.sk_wgs > 0)
        hipLaunchKernelGGL((gemm_f32t_kernel<MT, NT, WM, WN, ST, true>), grid, dim3(WM * WN * 64), 0, stream, p);
    else
        hipLaunchKernelGGL((gemm_f32t_kernel<MT, NT, WM, WN, ST, false>), grid, dim3(WM * WN * 64), 0, stream, p);
    return hipGetLastError();
}

constexpr int lds_f32(int mt, int nt, int kt, int st, int ks, int lay) {
    return (ks * st * (mt * (lay == LAYOUT_PAD ? kt + 4 : kt) + kt * (nt + 4)) > (ks - 1) * mt * nt
                ? ks * st * (mt * (lay == LAYOUT_PAD ? kt + 4 : kt) + kt * (nt + 4))
                : (ks - 1) * mt * nt) * 4;
}
constexpr int default_layout_f32(int kt) { return kt == 16 ? LAYOUT_SWIZZLE : LAYOUT_PAD; }

#define NNJIT_F32_VARIANT(MT, NT, KT, WM, WN, MF, ST, PF, KS, VEC)                                        \
    {"gemm_f32_" #MT "x" #NT "x" #KT "_w" #WM "x" #WN "_m" #MF "_s" #ST "_p" #PF "_k" #KS "_v" #VEC,             \
     FAM_GEMM_F32, MF, (MF == 32 ? 2 : 4), MT, NT, KT, WM, WN, ST, PF, KS, (VEC ? 16 : 4), 0, 0,               \
     KS * WM * WN * 64, lds_f32(MT, NT, KT, ST, KS, default_layout_f32(KT)),                                  \
     est_regs_f32(MT, NT, KT, WM, WN, MF, PF), (const void *)&gemm_f32_kernel<MT, NT, KT, WM, WN, MF, ST, PF, KS, VEC>, \
     &launch_gemm_f32<MT, NT, KT, WM, WN, MF, ST, PF, KS, VEC>, 0, default_layout_f32(KT), 0}

// Primitive-probe variants: a configuration of the list below with one
// primitive changed -- the A slab layout (LAY) or a rolled K-step loop
// (ROLL) -- for the offline one-variable-at-a-time benchmark.
#define NNJIT_F32P_VARIANT(MT, NT, KT, WM, WN, MF, ST, PF, KS, LAY, ROLL, TAG)                               \
    {"gemm_f32_" #MT "x" #NT "x" #KT "_w" #WM "x" #WN "_m" #MF "_s" #ST "_p" #PF "_k" #KS "_vtrue_" TAG,         \
     FAM_GEMM_F32, MF, (MF == 32 ? 2 : 4), MT, NT, KT, WM, WN, ST, PF, KS, 16, 0, 0,                           \
     KS * WM * WN * 64, lds_f32(MT, NT, KT, ST, KS, LAY), est_regs_f32(MT, NT, KT, WM, WN, MF, PF),            \
     (const void *)&gemm_f32_kernel<MT, NT, KT, WM, WN, MF, ST, PF, KS, true, LAY, ROLL>,                     \
     &launch_gemm_f32<MT, NT, KT, WM, WN, MF, ST, PF, KS, true, LAY, ROLL>, 0, LAY, ROLL}

#define NNJIT_F32P_LIST(X) \
    X(128, 128, 16, 2, 2, 32, 2, 2, 1, LAYOUT_PAD, false, "lpad") \
    X(128, 128, 16, 2, 2, 32, 2, 2, 1, LAYOUT_PLAIN, false, "lplain") \
    X(128, 128, 16, 2, 2, 32, 2, 2, 1, LAYOUT_SWIZZLE, true, "rolled") \
    X(64, 64, 16, 2, 2, 32, 2, 2, 1, LAYOUT_PAD, false, "lpad") \
    X(64, 64, 16, 2, 2, 32, 2, 2, 1, LAYOUT_PLAIN, false, "lplain") \
    X(64, 64, 32, 2, 2, 32, 2, 2, 1, LAYOUT_SWIZZLE, false, "lswz") \
    X(64, 64, 32, 2, 2, 32, 2, 2, 1, LAYOUT_PLAIN, false, "lplain") \
    X(64, 64, 32, 2, 2, 32, 2, 2, 1, LAYOUT_PAD, true, "rolled") \
    X(64, 64, 64, 2, 2, 32, 2, 2, 1, LAYOUT_SWIZZLE, false, "lswz") \
    X(64, 64, 64, 2, 2, 32, 2, 2, 1, LAYOUT_PAD, true, "rolled") \
    X(128, 128, 32, 2, 2, 32, 2, 2, 1, LAYOUT_SWIZZLE, false, "lswz") \
    X(128, 128, 32, 2, 2, 32, 2, 2, 1, LAYOUT_PLAIN, false, "lplain")

// Register estimate of the Table 1 formula Reg_thread = x0*r0 + r0*y0 + x0*y0
// for one lane: the accumulator tile (x0*y0 over 64 lanes), the A and B
// fragments of one K step (r0*y0, r0*x0), the global->LDS staging registers,
// and a fixed overhead for addresses and indices.
constexpr int est_regs_f32(int mt, int nt, int kt, int wm, int wn, int mf, int pf) {
    return (mt / wm) * (nt / wn) / 64 + 4 * ((mt / wm) / mf) + ((nt / wn) / mf) +
           pf * ((mt * kt + kt * nt) / (wm * wn * 64)) + 28;
}

// Wave-private variants: accumulators, one slab of A fragments (8 k) and B
// values, three registers of copy state per copy, and a fixed overhead.
constexpr int est_regs_f32w(int mt, int nt) {
    return (mt / 32) * (nt / 32) * 16 + (mt / 32) * 8 + (nt / 32) + 3 * (mt / 16 + 16 * nt / 256) + 24;
}
constexpr int lds_f32w(int mt, int nt, int ks, int st) {
    return ks * st * (mt * 64 + (16 / (256 / nt)) * (1024 + 16 * (256 / nt))) > ks * (mt / 32) * (nt / 32) * 16 * 256
               ? ks * st * (mt * 64 + (16 / (256 / nt)) * (1024 + 16 * (256 / nt)))
               : ks * (mt / 32) * (nt / 32) * 16 * 256;
}
#define NNJIT_F32W_VARIANT(MT, NT, KS, ST)                                                                   \
    {"gemm_f32w_" #MT "x" #NT "x16_k" #KS "_s" #ST, FAM_GEMM_F32, 32, 2, MT, NT, 16, 1, 1, ST, ST - 1, KS, 16,  \
     0, 0, KS * 64, lds_f32w(MT, NT, KS, ST), est_regs_f32w(MT, NT), (const void *)&gemm_f32w_kernel<MT, NT, KS, ST>, \
     &launch_gemm_f32w<MT, NT, KS, ST>, 1, LAYOUT_SWIZZLE, 0}

#define NNJIT_F32W_LIST(X) \
    X(64, 32, 4, 4) \
    X(64, 32, 8, 3) \
    X(32, 32, 4, 4) \
    X(32, 32, 8, 4) \
    X(32, 64, 4, 4) \
    X(64, 64, 4, 3) \
    X(64, 64, 4, 4) \
    X(128, 32, 4, 3) \
    X(32, 128, 4, 3)

#define NNJIT_F32W_INST(MT, NT, KS, ST) template __global__ void gemm_f32w_kernel<MT, NT, KS, ST>(GemmParams);
NNJIT_F32W_LIST(NNJIT_F32W_INST)

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
    X(128, 128, 32, 2, 2, 32, 2, 2, 1, true) \
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

// Shared-slab direct-copy variants: accumulators, one slab of fragments, the
// per-lane copy geometry (2 registers per copy) and a fixed overhead.
constexpr int est_regs_f32t(int mt, int nt, int wm, int wn) {
    return (mt / wm) * (nt / wn) / 64 + 8 * ((mt / wm) / 32) + 8 * ((nt / wn) / 32) +
           2 * ((mt * 64 + 64 * nt) / 1024 / (wm * wn)) + 32;
}
constexpr int lds_f32t(int mt, int nt, int st) { return st * (mt * 64 + 64 * nt); }
#define NNJIT_F32T_VARIANT(MT, NT, WM, WN, ST)                                                                \
    {"gemm_f32t_" #MT "x" #NT "x16_w" #WM "x" #WN "_s" #ST, FAM_GEMM_F32, 32, 2, MT, NT, 16, WM, WN, ST, ST - 1, \
     1, 16, 0, 0, WM * WN * 64, lds_f32t(MT, NT, ST), est_regs_f32t(MT, NT, WM, WN),                          \
     (const void *)&gemm_f32t_kernel<MT, NT, WM, WN, ST>, &launch_gemm_f32t<MT, NT, WM, WN, ST>, 1, LAYOUT_SWIZZLE, 0}

// The compiled shared-slab direct-copy configurations (16-byte aligned
// operands, Nt >= 64).
#define NNJIT_F32T_LIST(X) \
    X(256, 128, 4, 2, 3) \
    X(256, 128, 4, 2, 4) \
    X(128, 256, 2, 4, 4) \
    X(256, 256, 2, 4, 3) \
    X(256, 256, 4, 2, 3) \
    X(128, 128, 2, 2, 3) \
    X(128, 128, 2, 2, 4) \
    X(128, 128, 2, 4, 4) \
    X(128, 64, 2, 1, 4) \
    X(64, 128, 1, 2, 4) \
    X(64, 64, 2, 2, 4)

#define NNJIT_F32T_INST(MT, NT, WM, WN, ST)                                           \
    template __global__ void gemm_f32t_kernel<MT, NT, WM, WN, ST, false>(GemmParams); \
    template __global__ void gemm_f32t_kernel<MT, NT, WM, WN, ST, true>(GemmParams);
NNJIT_F32T_LIST(NNJIT_F32T_INST)

#define NNJIT_F32_INST(MT, NT, KT, WM, WN, MF, ST, PF, KS, VEC) \
    template __global__ void gemm_f32_kernel<MT, NT, KT, WM, WN, MF, ST, PF, KS, VEC>(GemmParams);
NNJIT_F32_LIST(NNJIT_F32_INST)
#define NNJIT_F32P_INST(MT, NT, KT, WM, WN, MF, ST, PF, KS, LAY, ROLL, TAG) \
    template __global__ void gemm_f32_kernel<MT, NT, KT, WM, WN, MF, ST, PF, KS, true, LAY, ROLL>(GemmParams);
NNJIT_F32P_LIST(NNJIT_F32P_INST)

#if !defined(__HIP_DEVICE_COMPILE__)
#define NNJIT_F32_ENTRY(...) NNJIT_F32_VARIANT(__VA_ARGS__),
#define NNJIT_F32W_ENTRY(...) NNJIT_F32W_VARIANT(__VA_ARGS__),
#define NNJIT_F32T_ENTRY(...) NNJIT_F32T_VARIANT(__VA_ARGS__),
#define NNJIT_F32P_ENTRY(...) NNJIT_F32P_VARIANT(__VA_ARGS__),
const Variant kGemmF32Variants[] = {NNJIT_F32_LIST(NNJIT_F32_ENTRY) NNJIT_F32W_LIST(NNJIT_F32W_ENTRY)
                                        NNJIT_F32T_LIST(NNJIT_F32T_ENTRY) NNJIT_F32P_LIST(NNJIT_F32P_ENTRY)};
const int kNumGemmF32Variants = sizeof(kGemmF32Variants) / sizeof(kGemmF32Variants[0]);
#endif

}  // namespace nnjit
