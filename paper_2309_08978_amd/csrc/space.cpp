// Configurations, the Table 1 resource model and the lite-space builder of
// the paper's device-guided space building (Sec. 5.2), on one CDNA4 CU.
// Host-only: no HIP runtime calls.
#include "space.h"

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdio>

namespace nnjit {

static const Variant *variant_at(int gi) {
    if (gi < kNumGemmF32Variants) return &kGemmF32Variants[gi];
    gi -= kNumGemmF32Variants;
    if (gi < kNumGemmF16Variants) return &kGemmF16Variants[gi];
    gi -= kNumGemmF16Variants;
    if (gi < kNumGemvVariants) return &kGemvVariants[gi];
    gi -= kNumGemvVariants;
    return &kGemvQ4Variants[gi];
}

int total_variants() { return kNumGemmF32Variants + kNumGemmF16Variants + kNumGemvVariants + kNumGemvQ4Variants; }

int variant_index(const Variant *v) {
    if (v >= kGemmF32Variants && v < kGemmF32Variants + kNumGemmF32Variants) return (int)(v - kGemmF32Variants);
    if (v >= kGemmF16Variants && v < kGemmF16Variants + kNumGemmF16Variants)
        return kNumGemmF32Variants + (int)(v - kGemmF16Variants);
    if (v >= kGemvVariants && v < kGemvVariants + kNumGemvVariants)
        return kNumGemmF32Variants + kNumGemmF16Variants + (int)(v - kGemvVariants);
    return kNumGemmF32Variants + kNumGemmF16Variants + kNumGemvVariants + (int)(v - kGemvQ4Variants);
}

const std::vector<int> &gemm_splits() {
    static const std::vector<int> s = {1, 2, 4, 8, 16};
    return s;
}
const std::vector<int> &gemv_splits() {
    static const std::vector<int> s = {1, 2, 4, 8, 16, 32, 64, 128};
    return s;
}

int family_dtype(int family) {
    return (family == FAM_GEMM_F16 || family == FAM_GEMV_F16 || family == FAM_GEMV_Q4) ? NNJIT_F16 : NNJIT_F32;
}
bool family_is_gemv(int family) { return family == FAM_GEMV_F32 || family == FAM_GEMV_F16; }
bool family_is_q4(int family) { return family == FAM_GEMV_Q4; }
int family_of(int kind, int dtype) {
    if (kind == NNJIT_KIND_GEMV_Q4) return FAM_GEMV_Q4;
    if (kind == NNJIT_KIND_GEMV) return dtype == NNJIT_F16 ? FAM_GEMV_F16 : FAM_GEMV_F32;
    return dtype == NNJIT_F16 ? FAM_GEMM_F16 : FAM_GEMM_F32;
}
const char *family_name(int family) {
    switch (family) {
    case FAM_GEMM_F32: return "gemm_f32";
    case FAM_GEMM_F16: return "gemm_f16";
    case FAM_GEMV_F32: return "gemv_f32";
    case FAM_GEMV_F16: return "gemv_f16";
    case FAM_GEMV_Q4: return "gemv_q4";
    default: return "?";
    }
}

const std::vector<Config> &configs() {
    static const std::vector<Config> all = [] {
        std::vector<Config> out;
        const int nv = total_variants();
        for (int gi = 0; gi < nv; ++gi) {
            const Variant *v = variant_at(gi);
            static const std::vector<int> no_split = {1};
            const std::vector<int> &splits =
                family_is_q4(v->family) ? no_split : family_is_gemv(v->family) ? gemv_splits() : gemm_splits();
            for (int s : splits) out.push_back(Config{(int)out.size(), v, s});
            if (has_stream_k(*v)) out.push_back(Config{(int)out.size(), v, kStreamK});
        }
        return out;
    }();
    return all;
}

nnjit_device_limits mi355x_limits() {
    nnjit_device_limits d;
    d.num_cus = 256;
    d.simds_per_cu = 4;
    d.vgprs_per_lane = 512;
    d.vgpr_granule = 8;
    d.max_waves_per_simd = 8;
    d.wave_size = 64;
    d.lds_per_cu = 163840;
    d.lds_per_wg = 163840;
    d.max_threads_per_wg = 1024;
    return d;
}

// Table 1 of the paper, on one compute unit ("core"):
//   Reg_thread   -> VGPR+AGPR per lane (measured from the compiled kernel, or
//                   the estimate inflated by the relaxation ratio)
//   L1_block     -> LDS bytes of the workgroup (the C tile lives in registers)
//   Thread_block -> workgroup size;  Warp_block -> waves of 64 lanes
//   Block_core   =  min(RegLimit, L1Limit, WarpLimit)
// RegLimit counts whole waves: a SIMD holds floor(512 / regs) waves (regs
// rounded up to the allocation granule), at most max_waves_per_simd.
nnjit_resources resources_of(const Variant &v, const nnjit_device_limits &d, int measured_regs) {
    nnjit_resources r{};
    const int regs = measured_regs >= 0 ? measured_regs : (int)std::ceil(v.est_regs / kRelaxation);
    r.regs_per_lane = regs;
    r.regs_measured = measured_regs >= 0 ? 1 : 0;
    r.lds_per_wg = v.lds_bytes;
    r.threads_per_wg = v.threads;
    r.waves_per_wg = (v.threads + d.wave_size - 1) / d.wave_size;
    const int gran = d.vgpr_granule > 0 ? d.vgpr_granule : 1;
    const int g = ((std::max(regs, 1) + gran - 1) / gran) * gran;
    const int wps = std::min(d.max_waves_per_simd, d.vgprs_per_lane / g);
    r.reg_limit = (d.simds_per_cu * wps) / r.waves_per_wg;
    r.lds_limit = v.lds_bytes > 0 ? (int)std::min<int64_t>(d.lds_per_cu / v.lds_bytes, 1 << 20) : (1 << 20);
    r.wave_limit = (d.simds_per_cu * d.max_waves_per_simd) / r.waves_per_wg;
    r.wg_per_cu = std::min(r.reg_limit, std::min(r.lds_limit, r.wave_limit));
    return r;
}

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
static int64_t pow2ceil(int64_t x) {
    int64_t p = 1;
    while (p < x) p <<= 1;
    return p;
}

bool has_stream_k(const Variant &v) { return v.family == FAM_GEMM_F32 && v.direct_copy && v.kslices == 1; }

Geometry geometry_of(const Config &c, int64_t batch, int64_t M, int64_t N, int64_t K, int64_t sk_wgs) {
    Geometry g;
    const Variant &v = *c.v;
    g.split = c.split == kStreamK ? 1 : c.split;
    if (c.split == kStreamK && batch == 1 && K > 0 && sk_wgs > 0) {
        g.stream_k = true;
        g.tiles_m = (int)ceil_div(std::max<int64_t>(M, 1), v.mt);
        g.tiles_n = (int)ceil_div(std::max<int64_t>(N, 1), v.nt);
        g.nslab = (int)ceil_div(K, v.kt);
        g.units = (int64_t)g.tiles_m * g.tiles_n * g.nslab;
        g.kchunk = (int)(g.nslab * (int64_t)v.kt);
        g.wgs = std::max<int64_t>(1, std::min<int64_t>(sk_wgs, g.units));
        g.ws_floats = 2 * g.wgs * (int64_t)v.mt * v.nt;
        return g;
    }
    if (family_is_q4(v.family)) {
        // one workgroup per nt output rows, no split (batch carries the group size)
        g.group = std::max<int64_t>(1, batch);
        g.tiles_m = 1;
        g.tiles_n = (int)ceil_div(std::max<int64_t>(N, 1), v.nt);
        g.kchunk = (int)std::max<int64_t>(K, 1);
        g.split = 1;
        g.wgs = g.tiles_n;
        g.ws_floats = 0;
        return g;
    }
    if (!family_is_gemv(v.family)) {
        g.tiles_m = (int)ceil_div(std::max<int64_t>(M, 1), v.mt);
        g.tiles_n = (int)ceil_div(std::max<int64_t>(N, 1), v.nt);
        const int64_t per = ceil_div(std::max<int64_t>(K, 1), g.split);
        g.kchunk = (int)(ceil_div(per, v.kt) * v.kt);
        const int64_t tiles = batch * g.tiles_m * (int64_t)g.tiles_n;
        g.wgs = tiles * g.split;
        g.ws_floats = g.split > 1 ? (int64_t)g.split * batch * std::max<int64_t>(M, 1) * std::max<int64_t>(N, 1) : 0;
    } else {
        g.tiles_m = 1;
        g.tiles_n = (int)ceil_div(std::max<int64_t>(N, 1), v.nt);
        g.kchunk = (int)std::max<int64_t>(1, ceil_div(std::max<int64_t>(K, 1), c.split));
        g.wgs = (int64_t)g.tiles_n * c.split;
        g.ws_floats = c.split > 1 ? (int64_t)c.split * std::max<int64_t>(N, 1) : 0;
    }
    return g;
}

const std::vector<ConsistentSetting> &consistent_settings() {
    static const std::vector<ConsistentSetting> t = {
#include "consistent.inc"
    };
    return t;
}

int primitive_value(const Variant &v, int primitive) {
    switch (primitive) {
    case PRIM_DIRECT: return v.direct_copy;
    case PRIM_LAYOUT: return v.lds_layout;
    case PRIM_UNROLL: return v.rolled;
    case PRIM_STAGES: return v.stages;
    case PRIM_PREFETCH: return v.prefetch;
    case PRIM_KT: return v.kt;
    case PRIM_MFMA: return v.mfma_m;
    case PRIM_VEC: return v.vec_bytes;
    default: return -1;
    }
}

// Do u and v differ in nothing but `primitive` (for the staging primitive:
// the same tile hierarchy, instruction shape and load width)?  The groups
// the offline microbenchmark compares.
static bool same_group(const Variant &u, const Variant &v, int primitive) {
    if (u.family != v.family || u.mfma_m != v.mfma_m || u.mfma_k != v.mfma_k || u.mt != v.mt || u.nt != v.nt ||
        u.kt != v.kt || u.wm != v.wm || u.wn != v.wn || u.vec_bytes != v.vec_bytes)
        return false;
    if (primitive == PRIM_DIRECT) return true;
    for (int q : {PRIM_DIRECT, PRIM_LAYOUT, PRIM_UNROLL, PRIM_STAGES, PRIM_PREFETCH, PRIM_KT, PRIM_MFMA, PRIM_VEC})
        if (q != primitive && primitive_value(u, q) != primitive_value(v, q)) return false;
    return u.kslices == v.kslices;
}

// A variant is excluded when a fixed (consistent) setting differs from its
// own and the compiled set holds its twin with the fixed setting: the
// primitive is fixed where the choice exists, not for variants the
// benchmark never compared.
bool follows_consistent(const Variant &v) {
    for (const ConsistentSetting &c : consistent_settings()) {
        if (c.family != v.family) continue;
        if (!(v.direct_copy ? c.direct_copy : c.reg_staged)) continue;
        if (primitive_value(v, c.primitive) == c.value) continue;
        for (const Config &u : configs())
            if (u.split == 1 && primitive_value(*u.v, c.primitive) == c.value && same_group(*u.v, v, c.primitive))
                return false;
    }
    return true;
}

namespace {
struct Cand {
    int id;
    nnjit_resources r;
    double eff;      // fill of the last wave of workgroups
    int64_t area;    // macro-tile area (GEMM) or columns x rows per pass (GEMV)
    int split;
};
}  // namespace

LiteResult lite_space(const Shape &s, const nnjit_device_limits &d, const std::vector<int> *measured_regs,
                      const std::vector<int> *spills) {
    LiteResult out;
    const int fam = family_of(s.kind, s.dtype);
    const bool gemv = family_is_gemv(fam);
    const bool q4 = family_is_q4(fam);
    const int V = vec_elems(s.dtype);
    const bool vec_ok = q4 ? (s.batch % 32 == 0) : gemv ? (s.N % V == 0) : (s.K % V == 0 && s.N % V == 0);

    // size of the unpruned parameter space over the same axes
    if (q4) {
        out.n_naive = 4 /*rows per wave*/ * 3 /*threads*/ * 3 /*K-slices*/ * 2 /*blocks in flight*/;
    } else if (!gemv) {
        const int64_t kt_choices = fam == FAM_GEMM_F32 ? 2 : 1;
        out.n_naive = 2 /*mfma*/ * 5 /*Mt*/ * 5 /*Nt*/ * kt_choices * 3 /*WM*/ * 3 /*WN*/ * 2 /*stages*/ *
                      (int64_t)gemm_splits().size();
    } else {
        out.n_naive = 3 /*L*/ * 5 /*threads*/ * 4 /*U*/ * (int64_t)gemv_splits().size();
    }

    std::vector<Cand> cands, unfit;  // unfit: pass the resource heuristics, fail the shape fit (split 1 only)
    std::vector<Cand> off_cands, off_unfit;  // the same, with a setting the consistent-primitive table excludes
    for (const Config &c : configs()) {
        const Variant &v = *c.v;
        if (v.family != fam) continue;
        ++out.n_enumerated;
        if ((v.vec_bytes == 16) != vec_ok) continue;  // vector loads only where the shape allows them
        const bool consistent = follows_consistent(v);
        const int gi = variant_index(&v);
        if (spills && gi < (int)spills->size() && (*spills)[gi]) continue;
        const int mregs = (measured_regs && gi < (int)measured_regs->size()) ? (*measured_regs)[gi] : -1;
        const nnjit_resources r = resources_of(v, d, mregs);
        if (r.threads_per_wg > d.max_threads_per_wg) continue;                // heuristic 5
        if (r.lds_per_wg > d.lds_per_wg) continue;                            // heuristic 6
        if (r.wg_per_cu < 1) continue;

        const int64_t slots = (int64_t)d.num_cus * r.wg_per_cu;
        const Geometry g = geometry_of(c, s.batch, s.M, s.N, s.K, slots);
        Cand cd;
        cd.id = c.id;
        cd.r = r;
        const int64_t waves = ceil_div(std::max<int64_t>(g.wgs, 1), slots);
        cd.eff = (double)g.wgs / (double)(waves * slots);
        cd.area = (int64_t)v.mt * v.nt * ((gemv || q4) ? v.kt : 1);
        cd.split = c.split;
        bool fit = true;
        if (q4) {
            // no workgroup wider than the (power-of-two rounded) output count;
            // K-slices and blocks in flight only where K has the blocks for them
            if (v.nt > std::max<int64_t>(8, pow2ceil(s.N))) fit = false;
            const int64_t nblk = std::max<int64_t>(1, ceil_div(s.K, v.kt));
            if (v.kslices > 1 && nblk < v.kslices) fit = false;
            if (v.unroll > 1 && ceil_div(nblk, v.kslices) < v.unroll) fit = false;
        } else if (!gemv) {
            // shape fit: no macro tile wider than the (power-of-two rounded) matrix
            if (v.mt > std::max<int64_t>(16, pow2ceil(s.M)) || v.nt > std::max<int64_t>(16, pow2ceil(s.N))) fit = false;
            const int64_t tiles = s.batch * g.tiles_m * (int64_t)g.tiles_n;
            if (c.split == kStreamK) {
                // stream-K: only where the tiles leave the last wave of
                // workgroups short, with at least four K slabs per workgroup
                if (!g.stream_k || g.units < 4 * g.wgs) continue;
                const int64_t tw = ceil_div(tiles, slots);
                if ((double)tiles / (double)(tw * slots) >= 0.95) continue;
                cd.eff = 1.0;
            }
            // K groups inside a workgroup pay off only while the chip has
            // few workgroups (fewer than two per CU)
            if (v.kslices > 1 && tiles * c.split >= 2LL * d.num_cus) continue;
            if (c.split > 1) {
                // split K only to fill the CUs: keep the smallest power of two
                // that gives every CU a workgroup, and twice that
                if (tiles >= d.num_cus) continue;
                int64_t sfill = 1;
                while (tiles * sfill < d.num_cus) sfill <<= 1;
                // a workgroup with K groups needs half the split for the same waves
                const int64_t lo = v.kslices > 1 ? std::max<int64_t>(1, sfill / 2) : sfill;
                if (c.split < lo || c.split > 2 * sfill) continue;
                // over-split: more than two waves of workgroups, unless they
                // form whole waves (at most four)
                const int64_t wgs = tiles * c.split;
                if (wgs > 2 * slots && !(wgs % slots == 0 && wgs <= 4 * slots)) continue;
                if (s.K < 2LL * c.split * v.kt) continue;    // at least two K slabs per split
            }
        } else {
            if (v.nt > std::max<int64_t>(64, pow2ceil(s.N))) fit = false;
            const int rows_per_pass = v.kt;
            if (c.split > 1) {
                if (g.kchunk < rows_per_pass) continue;  // every split gets at least one pass of rows
                int smax = 1;
                for (int sp : gemv_splits())
                    if (ceil_div(std::max<int64_t>(s.K, 1), sp) >= rows_per_pass) smax = sp;
                // split only to fill the CUs: the smallest power of two that
                // gives every CU a workgroup, and twice that (or the largest
                // split K allows)
                if (g.tiles_n >= d.num_cus) continue;
                int64_t sfill = 1;
                while (g.tiles_n * sfill < d.num_cus) sfill <<= 1;
                if ((c.split < sfill || c.split > 2 * sfill) && c.split != smax) continue;
                if (g.wgs > 4 * slots) continue;                                  // over-split
                if (g.wgs < d.num_cus / 2 && c.split != smax) continue;           // under-filled
                // Little's law: bytes in flight per CU must cover HBM latency
                const int64_t wg_here = std::min<int64_t>(r.wg_per_cu, ceil_div(g.wgs, d.num_cus));
                if (wg_here * v.threads * (int64_t)v.unroll * 16 < 8192 && c.split != smax) continue;
            }
        }
        if (fit) (consistent ? cands : off_cands).push_back(cd);
        else if (c.split == 1) (consistent ? unfit : off_unfit).push_back(cd);
    }
    // settings fixed offline (consistent primitives) prune the rest, unless
    // nothing would be left (e.g. element-load shapes when 16-byte loads are
    // the fixed setting)
    if (cands.empty() && unfit.empty()) {
        cands.swap(off_cands);
        unfit.swap(off_unfit);
    }
    // the shape fit never empties the space: tiny shapes fall back to the
    // unsplit configurations that passed the resource heuristics
    if (cands.empty()) cands = unfit;

    // heuristic 7: keep register-bound candidates (Block_core == RegLimit),
    // relaxed when too few survive.  A direct-copy variant keeps its staging
    // (the slabs in flight, a register term of Table 1 for the others) in
    // LDS, so for it the bound that plays this role is L1Limit.
    std::vector<Cand> kept;
    for (const Cand &c : cands) {
        const bool direct = configs()[c.id].v->direct_copy != 0;
        if (c.r.wg_per_cu == (direct ? c.r.lds_limit : c.r.reg_limit)) kept.push_back(c);
    }
    if ((int)kept.size() < kMinSurvivors) kept = cands;

    // evaluation order: most workgroups per CU first, then fuller last wave,
    // larger tile, smaller split, lower id -- within each staging kind
    // (registers / LDS direct copies), the two orders merged in turn so that
    // the cap below never drops one kind wholesale
    auto before = [](const Cand &a, const Cand &b) {
        if (a.r.wg_per_cu != b.r.wg_per_cu) return a.r.wg_per_cu > b.r.wg_per_cu;
        if (std::fabs(a.eff - b.eff) > 1e-9) return a.eff > b.eff;
        if (a.area != b.area) return a.area > b.area;
        if (a.split != b.split) return a.split < b.split;
        return a.id < b.id;
    };
    std::vector<Cand> by_kind[2];
    for (const Cand &c : kept) by_kind[configs()[c.id].v->direct_copy != 0 ? 1 : 0].push_back(c);
    for (auto &v : by_kind) std::stable_sort(v.begin(), v.end(), before);
    std::vector<Cand> order;
    for (size_t i = 0; i < std::max(by_kind[0].size(), by_kind[1].size()); ++i)
        for (auto &v : by_kind)
            if (i < v.size()) order.push_back(v[i]);
    // the lite space is the head of that order: at most kMaxTimed candidates
    // are ever evaluated on the device
    for (const Cand &c : order) {
        if ((int)out.ids.size() >= kMaxTimed) break;
        out.ids.push_back(c.id);
    }
    return out;
}

}  // namespace nnjit
