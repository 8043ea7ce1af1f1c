// Configurations, the Table 1 resource model and the lite-space builder.
// Host-only code: nothing here calls the HIP runtime.
#pragma once

#include <cstdint>
#include <vector>

#include "internal.h"
#include "../../include/nnjit.h"

namespace nnjit {

// A configuration = a compiled variant + a split-K factor.  Its id is its
// index in configs().
struct Config {
    int id;
    const Variant *v;
    int split;
};

const std::vector<Config> &configs();

// Split-K factors considered per kind (powers of two, heuristic 2).
const std::vector<int> &gemm_splits();
const std::vector<int> &gemv_splits();

int family_dtype(int family);       // NNJIT_F32 / NNJIT_F16
bool family_is_gemv(int family);    // fp32 / fp16 GEMV (not the 4-bit one)
bool family_is_q4(int family);      // 4-bit weight-only GEMV
int family_of(int kind, int dtype);  // family whose kernels run this kind/dtype
const char *family_name(int family);

// Elements of 16 bytes for a dtype (the vector width of heuristic 1).
inline int vec_elems(int dtype) { return dtype == NNJIT_F16 ? 8 : 4; }

// MI355X defaults for host-only use.
nnjit_device_limits mi355x_limits();

// Table 1 of the paper on one CDNA4 compute unit.  measured_regs < 0 means
// "not measured": the estimate is used, inflated by the relaxation ratio.
nnjit_resources resources_of(const Variant &v, const nnjit_device_limits &d, int measured_regs);

constexpr double kRelaxation = 0.9;  // share of the register file the estimate may claim
constexpr int kMaxTimed = 96;        // size cap of a lite space (candidates timed per shape at most)
constexpr int kMinSurvivors = 8;     // heuristic 7 is relaxed below this many

// Primitives whose setting the offline microbenchmark may fix for a whole
// family (the paper's consistent primitives, Sec. 5.1).
enum Primitive { PRIM_DIRECT, PRIM_LAYOUT, PRIM_UNROLL, PRIM_STAGES, PRIM_PREFETCH, PRIM_KT, PRIM_MFMA, PRIM_VEC };
struct ConsistentSetting {
    int family;
    int primitive;
    int value;
    int reg_staged;    // applies to register-staged variants
    int direct_copy;   // applies to direct-copy variants
};
// The table generated from the microbenchmark's stored measurement.
const std::vector<ConsistentSetting> &consistent_settings();
// The setting of a primitive in a variant (the integer the table stores).
int primitive_value(const Variant &v, int primitive);
// false if the variant has another setting of a primitive the table fixes.
bool follows_consistent(const Variant &v);

struct Shape {
    int kind;
    int dtype;
    int64_t batch, M, N, K;   // 4-bit GEMV: batch = group size, M = 1
};

struct LiteResult {
    std::vector<int> ids;       // survivors in evaluation order
    int n_enumerated = 0;       // compiled configurations of the family
    int64_t n_naive = 0;        // unpruned size of the parameter axes
};

// measured_regs: per-variant register counts of the compiled kernels for the
// family's variant table (empty = estimate); spills: per-variant flag.
LiteResult lite_space(const Shape &s, const nnjit_device_limits &d, const std::vector<int> *measured_regs,
                      const std::vector<int> *spills);

// The split value of a stream-K configuration (see GemmParams): the K slabs
// of all tiles cut evenly over one workgroup per resident slot.
constexpr int kStreamK = 0;
// Variants that have a stream-K configuration (fp32 shared-slab direct copy).
bool has_stream_k(const Variant &v);

// Launch geometry of a configuration for a shape.
struct Geometry {
    int tiles_m = 0, tiles_n = 0;  // GEMM tiles per batch slice (GEMV: segs in tiles_n)
    int split = 1;                 // split-K factor of the launch (1 for stream-K)
    int kchunk = 0;
    int64_t wgs = 0;               // workgroups over the whole launch
    int64_t ws_floats = 0;         // split-K partial storage (S x batch x M x N floats; stream-K 2 x wgs x Mt x Nt)
    int64_t group = 0;             // 4-bit GEMV: the group size
    bool stream_k = false;
    int nslab = 0;                 // stream-K: K slabs per tile
    int64_t units = 0;             // stream-K: tiles x nslab
};
// sk_wgs: the workgroups a stream-K configuration launches (resident slots of
// the device, CUs x workgroups per CU); unused by other configurations.  A
// stream-K configuration on a batch > 1 or K == 0 shape runs tiled (split 1).
Geometry geometry_of(const Config &c, int64_t batch, int64_t M, int64_t N, int64_t K, int64_t sk_wgs = 0);

// Index of a variant inside its family table (used to look up measured data).
int variant_index(const Variant *v);
int total_variants();

}  // namespace nnjit
