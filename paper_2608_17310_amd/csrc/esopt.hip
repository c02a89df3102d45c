// ES parameter path for MI355X (gfx950): perturb / restore / fused N-member
// update / reward z-score over a list of bf16 tensors, behind the C ABI of
// include/esopt.h.
//
// Method (arXiv 2608.17310): Section 3 (perturb theta + sigma eps_i, revert
// by subtraction, z-score rewards, theta += (alpha/G) sum zhat_i eps_i, noise
// regenerated from seeds), Section 3.1 (cosine sigma schedule), Appendix C.1
// (1/(G sigma) estimator), Appendix D.6 (order of apply / evaluate / revert /
// regenerate).
//
// Layout and launch shape:
//   * A plan cuts every tensor into tiles of T x U x 8 elements (T lanes per
//     workgroup, U 8-element groups per lane; by default 1024 x 8 x 8 =
//     65536 elements, 128 KB): full tiles on tile-sized boundaries of the
//     address space, then tail tiles (each tensor's head and remainder, or
//     every tile of an unaligned tensor), each described by a 32-byte
//     descriptor.  One launch covers the whole parameter list: a grid of
//     (CUs x WGs-per-CU) workgroups strides over the full tiles, then the
//     tails, reading one descriptor per tile with a scalar load, so a tile's
//     tensor, address and noise identity are wave-uniform.
//   * Within a tile, lane l of group slot u owns elements
//     elem0 + 8 (u * T + l) .. +7: one 16-byte load and one 16-byte store, 64
//     lanes covering 1 KB contiguous per instruction.  Its two Philox calls
//     are the quads 2 g and 2 g + 1 of that group (tiles start at multiples
//     of 8 elements); no tile crosses a multiple of 2^34 elements, so the
//     counter's high word is uniform per tile.
//   * Perturb is HBM-bound: one 1024-lane workgroup per CU streams 128 KB
//     tiles; the loads of its next tile are issued before the current tile's
//     arithmetic (software pipelining), and each tile's stores leave in one
//     burst after all its arithmetic.  The update is VALU-bound (N noise
//     streams per element): eight workgroups per CU keep every wave slot
//     busy, one 8-element group per lane at a time with the next group's
//     load in flight.  Both shapes were chosen by sweeping on MI355X.  Swap
//     is the perturb kernel with two streams and a bf16 rounding between
//     them.
//   * The quantized path (int8 codes, es_quant.hpp; fp8 E4M3 codes,
//     es_fp8.hpp) has a tensor table searched per tile and tiles of 16-code
//     groups; all its passes are VALU-bound and use the update's shape.
//   * Perturb/restore read and write each parameter once (4 bytes of HBM
//     traffic per parameter).  The update regenerates the noise of all
//     distinct member seeds for the same 8 elements in registers,
//     accumulates sum_d w_d eps_d in binary32, and then does the single
//     read-modify-write, so its HBM traffic does not depend on N.
//   * Tail tiles take a bounds-checked path with identical arithmetic:
//     16-byte accesses for whole groups of an aligned tensor, 2-byte accesses
//     for a partial group or an unaligned tensor.
//   * Blocks of row-major tensors that are not one contiguous range (column
//     shards) are tiled by address like tensors; their tiles carry a row map
//     from the element's place in the block to its whole-tensor index, the
//     noise index, and run in a second launch of the same kernels
//     instantiated with it (kRows).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstddef>
#include <cstring>
#include <atomic>
#include <mutex>
#include <new>
#include <string>
#include <type_traits>
#include <limits>
#include <unordered_map>
#include <vector>
#include <algorithm>

#include "../../include/esopt.h"
#include "es_fp8.hpp"
#include "es_noise.hpp"
#include "es_quant.hpp"
#include "es_table.hpp"

namespace {

constexpr int kAuxBlock = 256;              // lanes per workgroup of the small kernels
constexpr int kGroupElems = 8;              // bf16 per lane-group (one 16-byte access)
// Default tile shape and grids (measured on MI355X; see the launch-shape
// notes above).  The update is VALU-bound and wants every wave slot filled;
// perturb is HBM-bound and wants large contiguous per-CU streams.
constexpr int kDefaultThreads = 1024;
constexpr int kDefaultGroups = 8;
constexpr int kDefaultPerturbWgPerCu = 1;
constexpr int kDefaultUpdateWgPerCu = 8;
constexpr int kDefaultQGroups = 4;          // int8 tiles: 1024 x 4 x 16 codes (64 KB)
constexpr double kSqrt2Ln2Double = 1.1774100225154746910;   // sqrt(2 ln 2)

// Tile descriptor.  A plan lists its tiles in runs, indexed by tile number:
// full tiles first (kThreads * kU * 8 elements of one tensor, starting on a
// tile-sized boundary of the address space), then tail tiles (the part of a
// tensor before its first such boundary, the part after its last full tile,
// or every tile of a tensor whose base is not 16-byte aligned); the tiles of
// strided blocks (es_plan_create_blocks) follow in two more runs of the same
// kinds, each with a row map (DevRows), and are passed over in a second
// launch.  A workgroup reads one descriptor per tile with a single scalar
// load and no search (searching a per-tensor table is a chain of dependent
// scalar loads).
// Full tiles aligned to the address space, not to their tensor's base: with
// hundreds of tensors at unrelated offsets, tiles at mixed offsets streamed
// ~4 % slower.  32 bytes per 65 536-element tile.
struct DevTile {
    uint16_t* data;                         // the tensor's base
    uint64_t elem0;                         // the tile's first element in its tensor
    uint64_t limit;                         // one past the last element a tail tile may touch
    uint32_t tensor_id;
    uint32_t aligned16;                     // base 16-byte aligned: whole groups 16-byte accesses
};
static_assert(sizeof(DevTile) == 32, "tile descriptor layout");

// Row map of a tile of a strided block (es_block_t with rows > 1 and
// cols < row_len): the block is cut into pieces of whole rows, each tiled by
// address as a tensor of its own, so a tile's element index e is local to
// its piece (e < 2^31), and local element e is whole-tensor element
//   n0 + e + (e / cols) (row_len - cols),
// n0 being the piece's first whole-tensor index.  cols is a multiple of 8, so
// a group of 8 never spans two rows and its elements keep consecutive
// indices (one quad pair).  The row division is a multiply-high and a shift
// and skip = row_len - cols is below 2^32, so the map costs one 32 x 32-bit
// multiply-add and a 64-bit add per group.  As with contiguous tiles, no tile
// spans a multiple of 2^34 whole-tensor elements (the host splits it there),
// so the counter's high word `hi` is the tile's, wave-uniform.  One entry per
// tile, beside its descriptor.
struct DevRows {
    uint64_t n0;
    uint32_t skip;                          // row_len - cols
    uint32_t magic, shift;                  // e / cols = mulhi(e, magic) >> shift
    uint32_t hi;                            // whole-tensor index >> 34, the same for the tile
    uint32_t pad[2];
};
static_assert(sizeof(DevRows) == 32, "row map layout");

// Whole-tensor index of local element e (< 2^31) under a row map; the host
// tests call this same function.
__host__ __device__ __forceinline__ uint64_t rows_index(uint64_t n0, uint32_t skip, uint32_t magic,
                                                        uint32_t shift, uint64_t e) {
    const uint32_t el = static_cast<uint32_t>(e);
    const uint32_t row = static_cast<uint32_t>((uint64_t(el) * magic) >> 32) >> shift;
    return n0 + (uint64_t(row) * skip + el);
}

struct MemberIn {                           // one population member, CSR order
    uint32_t reward_index;
    int32_t sign;
};
struct DistinctIn {                         // one distinct seed and its members
    uint32_t k0, k1;
    uint32_t first;
    uint32_t count;
};
struct Member {                             // merged weight of one distinct seed
    uint32_t k0, k1;
    float w_k;                              // weight times sqrt(2 ln 2)
    uint32_t pad;
};
struct UpdateHeader {
    uint32_t n_distinct;
    uint32_t n_live;                        // distinct seeds with w != 0
    int32_t status;                         // 1: non-finite reward, update skipped
    uint32_t pad;
};

// Plan scratch layout (bytes).
constexpr size_t kOffMembersIn = 0;
constexpr size_t kOffDistinctIn = kOffMembersIn + sizeof(MemberIn) * ES_MAX_MEMBERS;
constexpr size_t kOffMembers = kOffDistinctIn + sizeof(DistinctIn) * ES_MAX_MEMBERS;
constexpr size_t kOffHeader = kOffMembers + sizeof(Member) * ES_MAX_MEMBERS;
constexpr size_t kScratchBytes = kOffHeader + 256;

constexpr int kStageWords = 256;            // 1 KB of kernel arguments per launch
constexpr uint64_t kMaxLayoutTiles = uint64_t(1) << 22;   // es_tile_layout's bound
struct StageChunk {
    uint32_t words[kStageWords];
};

thread_local std::string g_last_error;

int fail(int code, const std::string& msg) {
    g_last_error = msg;
    return code;
}

int hip_fail(hipError_t e, const std::string& what) {
    return fail(ES_ERR_HIP, what + ": " + hipGetErrorString(e));
}

// A failure of call `name`: the message is formatted only here, so a call
// that succeeds builds no strings (no host allocation on its way).
int fail_in(int code, const char* name, const char* msg) {
    return fail(code, std::string(name) + ": " + msg);
}

// ------------------------------------------------------------------------
// Device code
// ------------------------------------------------------------------------

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
// Tile descriptors and tensor tables hold generic pointers; every parameter
// lives in global memory, and saying so lets the compiler use global_load /
// global_store (vector-memory counters only) instead of flat accesses.
#define ES_GLOBAL __attribute__((address_space(1)))

// Load the 8 bf16 of one group (packed in 4 words).  Fast path: one 16-byte
// load (nontemporal when kNT: the parameters are streamed once per pass).
// Checked path (tail tiles): the 16-byte load when the tensor is 16-byte
// aligned and the whole group lies below the bound `limit`, element-wise
// 2-byte loads below the bound otherwise.
template <bool kFast, bool kNT>
__device__ __forceinline__ void load_group(const uint16_t* __restrict__ p, uint64_t e,
                                           uint64_t limit, uint32_t raw[4], bool vec = false) {
    if (kFast || (vec && e + 8 <= limit)) {
        const ES_GLOBAL u32x4_t* a = (const ES_GLOBAL u32x4_t*)(p + e);
        const u32x4_t v = kNT ? __builtin_nontemporal_load(a) : *a;
        raw[0] = v.x; raw[1] = v.y; raw[2] = v.z; raw[3] = v.w;
    } else {
        const ES_GLOBAL uint16_t* g = (const ES_GLOBAL uint16_t*)p;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint32_t lo = (e + 2 * k < limit) ? g[e + 2 * k] : 0u;
            const uint32_t hi = (e + 2 * k + 1 < limit) ? g[e + 2 * k + 1] : 0u;
            raw[k] = lo | (hi << 16);
        }
    }
}

template <bool kFast, bool kNT>
__device__ __forceinline__ void store_group(uint16_t* __restrict__ p, uint64_t e, uint64_t limit,
                                            const uint32_t out[4], bool vec = false) {
    if (kFast || (vec && e + 8 <= limit)) {
        ES_GLOBAL u32x4_t* a = (ES_GLOBAL u32x4_t*)(p + e);
        const u32x4_t v = {out[0], out[1], out[2], out[3]};
        if constexpr (kNT) __builtin_nontemporal_store(v, a);
        else *a = v;
    } else {
        ES_GLOBAL uint16_t* g = (ES_GLOBAL uint16_t*)p;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (e + 2 * k < limit) g[e + 2 * k] = static_cast<uint16_t>(out[k] & 0xFFFFu);
            if (e + 2 * k + 1 < limit) g[e + 2 * k + 1] = static_cast<uint16_t>(out[k] >> 16);
        }
    }
}

// The binary32 master copies of a group's 8 elements (es_plan_set_master):
// element e's master sits at mb + 4 e, mb being the tile's master base.  A
// group that takes the 16-byte bf16 path has a 16-byte aligned master group
// (the masters are 16-byte aligned and laid out as their bf16 tensors), so it
// takes two 16-byte accesses; element-wise accesses below the bound otherwise.
typedef float f32x4_t __attribute__((ext_vector_type(4)));

template <bool kFast, bool kNT>
__device__ __forceinline__ void load_master(uintptr_t mb, uint64_t e, uint64_t limit, float m[8],
                                            bool vec = false) {
    if (kFast || (vec && e + 8 <= limit)) {
        const ES_GLOBAL f32x4_t* a = (const ES_GLOBAL f32x4_t*)(mb + 4 * e);
        const f32x4_t v0 = kNT ? __builtin_nontemporal_load(a) : a[0];
        const f32x4_t v1 = kNT ? __builtin_nontemporal_load(a + 1) : a[1];
        m[0] = v0.x; m[1] = v0.y; m[2] = v0.z; m[3] = v0.w;
        m[4] = v1.x; m[5] = v1.y; m[6] = v1.z; m[7] = v1.w;
    } else {
        const ES_GLOBAL float* g = (const ES_GLOBAL float*)mb;
#pragma unroll
        for (int k = 0; k < 8; ++k) m[k] = (e + k < limit) ? g[e + k] : 0.0f;
    }
}

template <bool kFast, bool kNT>
__device__ __forceinline__ void store_master(uintptr_t mb, uint64_t e, uint64_t limit,
                                             const float m[8], bool vec = false) {
    if (kFast || (vec && e + 8 <= limit)) {
        ES_GLOBAL f32x4_t* a = (ES_GLOBAL f32x4_t*)(mb + 4 * e);
        const f32x4_t v0 = {m[0], m[1], m[2], m[3]};
        const f32x4_t v1 = {m[4], m[5], m[6], m[7]};
        if constexpr (kNT) {
            __builtin_nontemporal_store(v0, a);
            __builtin_nontemporal_store(v1, a + 1);
        } else {
            a[0] = v0;
            a[1] = v1;
        }
    } else {
        ES_GLOBAL float* g = (ES_GLOBAL float*)mb;
#pragma unroll
        for (int k = 0; k < 8; ++k)
            if (e + k < limit) g[e + k] = m[k];
    }
}

// The Philox words of the 8 elements of the group starting at element 8 g:
// quads 2 g and 2 g + 1 (q_lo is even, so q_lo + 1 does not carry into q_hi).
__device__ __forceinline__ void group_words(uint32_t q_lo, uint32_t q_hi, uint32_t tensor_id,
                                            uint32_t k0, uint32_t k1, uint32_t w[8]) {
    const es::Words a = es::philox4x32_10(q_lo, q_hi, tensor_id, es::kDomainNoise, k0, k1);
    const es::Words b = es::philox4x32_10(q_lo + 1u, q_hi, tensor_id, es::kDomainNoise, k0, k1);
    w[0] = a.w0; w[1] = a.w1; w[2] = a.w2; w[3] = a.w3;
    w[4] = b.w0; w[5] = b.w1; w[6] = b.w2; w[7] = b.w3;
}

// x[k] += scale * eps_k for the 8 elements of a group, in binary32: each
// Box-Muller pair (words 2p, 2p+1) feeds elements 2p (cos) and 2p+1 (sin);
// scale_k = scale * sqrt(2 ln 2).
__device__ __forceinline__ void group_axpy(const uint32_t w[8], float scale_k, float x[8]) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        float t, c, sn;
        es::scaled_pair(w[2 * p], w[2 * p + 1], scale_k, t, c, sn);
        x[2 * p] = __builtin_fmaf(t, c, x[2 * p]);
        x[2 * p + 1] = __builtin_fmaf(t, sn, x[2 * p + 1]);
    }
}

// Noise streams applied by one perturb-style pass.  kM = 1: one stream,
// theta <- RNE(theta + c_0 eps_0) (perturb / restore).  kM = 2: two streams
// applied in turn with a bf16 rounding in between,
// theta <- RNE(RNE(theta + c_0 eps_0) + c_1 eps_1), which is es_restore of
// one member followed by es_perturb of the next, bit for bit, in one pass
// (swap).  kM = 3: the same with both streams on one key (an antithetic
// partner), whose noise is generated once.  coef_k = c sqrt(2 ln 2).
struct Streams {
    uint32_t k0[2], k1[2];
    float coef_k[2];
};

__device__ __forceinline__ void round_to_bf16(float x[8]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t b = es::pack_bf16x2(x[2 * k], x[2 * k + 1]);
        x[2 * k] = es::bf16_lo(b);
        x[2 * k + 1] = es::bf16_hi(b);
    }
}

// Apply the streams to one 8-element group in registers and pack to bf16.
// Each stream adds one FMA per element to the binary32 value.
template <int kM>
__device__ __forceinline__ void perturb_group(const uint32_t raw[4], uint64_t e, uint32_t q_hi,
                                              uint32_t tensor_id, const Streams& st,
                                              uint32_t out[4]) {
    float x[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        x[2 * k] = es::bf16_lo(raw[k]);
        x[2 * k + 1] = es::bf16_hi(raw[k]);
    }
    if constexpr (kM == 3) {
        uint32_t w[8];
        group_words(static_cast<uint32_t>(e >> 2), q_hi, tensor_id, st.k0[0], st.k1[0], w);
        float r[4], c[4], sn[4];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            r[p] = es::pair_radius(w[2 * p]);
            es::pair_angle(w[2 * p + 1], c[p], sn[p]);
        }
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            if (m == 1) round_to_bf16(x);
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                const float t = st.coef_k[m] * r[p];
                x[2 * p] = __builtin_fmaf(t, c[p], x[2 * p]);
                x[2 * p + 1] = __builtin_fmaf(t, sn[p], x[2 * p + 1]);
            }
        }
    } else {
#pragma unroll
        for (int m = 0; m < kM; ++m) {
            if (m > 0) round_to_bf16(x);
            uint32_t w[8];
            group_words(static_cast<uint32_t>(e >> 2), q_hi, tensor_id, st.k0[m], st.k1[m], w);
            group_axpy(w, st.coef_k[m], x);
        }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) out[k] = es::pack_bf16x2(x[2 * k], x[2 * k + 1]);
}

// A tile: up to kThreads * kU * 8 consecutive elements of one tensor, from
// element elem0 on; accesses of a tail tile stay below `limit`.  A tile of a
// strided block also carries its piece's row map (DevRows): its elements are
// then addressed by elem0 + ... and draw the noise of their whole-tensor
// index.  Every field is wave-uniform (scalar registers).
struct TileRef {
    uint16_t* data;
    uint64_t limit;
    uint64_t elem0;
    uint32_t tensor_id;
    uint32_t aligned16;
    uint64_t n0 = 0;                        // row map (strided blocks only)
    uint32_t skip = 0, magic = 0, shift = 0, hi = 0;
};

__device__ __forceinline__ TileRef tile_ref(const DevTile& d) {
    return TileRef{d.data, d.limit, d.elem0, d.tensor_id, d.aligned16};
}

__device__ __forceinline__ TileRef tile_ref(const DevTile& d, const DevRows& m) {
    return TileRef{d.data, d.limit, d.elem0, d.tensor_id, d.aligned16, m.n0, m.skip, m.magic,
                   m.shift, m.hi};
}

// Tile i of a launch: its descriptor, and with kRows its row map.
template <bool kRows>
__device__ __forceinline__ TileRef load_ref(const DevTile* __restrict__ tiles,
                                            const DevRows* __restrict__ rows, uint64_t i) {
    if constexpr (kRows) return tile_ref(tiles[i], rows[i]);
    else return tile_ref(tiles[i]);
}

// Noise index of the group starting at element e of a tile: e itself, or
// the whole-tensor index through the tile's row map.
template <bool kRows>
__device__ __forceinline__ uint64_t noise_index(const TileRef& r, uint64_t e) {
    if constexpr (kRows) return rows_index(r.n0, r.skip, r.magic, r.shift, e);
    else return e;
}

// The counter's high word (whole-tensor index >> 34), uniform over a tile.
template <bool kRows>
__device__ __forceinline__ uint32_t tile_high_word(const TileRef& r) {
    if constexpr (kRows) return r.hi;
    else return static_cast<uint32_t>(r.elem0 >> 34);
}

// Keep a prefetched descriptor in scalar registers: without this the
// compiler may drop it and load it again where it is used, exposing the
// load's latency there.  Placed after the work that hides the load, so the
// wait it implies costs nothing.
__device__ __forceinline__ void keep_in_sgprs(DevTile& d) {
    asm volatile("" : "+s"(d.data), "+s"(d.elem0), "+s"(d.tensor_id));
}
__device__ __forceinline__ void keep_in_sgprs(DevRows& m) {
    asm volatile("" : "+s"(m.n0), "+s"(m.skip), "+s"(m.magic), "+s"(m.shift), "+s"(m.hi));
}

template <int kThreads, int kU>
__device__ __forceinline__ void load_tile(const TileRef& r, uint32_t raw[kU][4]) {
#pragma unroll
    for (int u = 0; u < kU; ++u) {
        const uint64_t e = r.elem0 + uint64_t(u * kThreads + threadIdx.x) * kGroupElems;
        load_group<true, true>(r.data, e, r.limit, raw[u]);
    }
}

// Perturb a full tile whose groups are already in registers: every group is
// computed first and the tile's stores then leave in one burst.  On MI355X
// an in-place stream whose writes come in per-tile bursts sustains ~6.2 TB/s,
// against ~5.5 TB/s when each group's store is interleaved with the next
// group's arithmetic.
template <int kThreads, int kU, int kM, bool kRows>
__device__ __forceinline__ void perturb_loaded(const TileRef& r, uint32_t raw[kU][4],
                                               const Streams& st) {
    const uint32_t q_hi = tile_high_word<kRows>(r);
#pragma unroll
    for (int u = 0; u < kU; ++u) {
        const uint64_t e = r.elem0 + uint64_t(u * kThreads + threadIdx.x) * kGroupElems;
        uint32_t out[4];
        perturb_group<kM>(raw[u], noise_index<kRows>(r, e), q_hi, r.tensor_id, st, out);
#pragma unroll
        for (int k = 0; k < 4; ++k) raw[u][k] = out[k];
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < kU; ++u) {
        const uint64_t e = r.elem0 + uint64_t(u * kThreads + threadIdx.x) * kGroupElems;
        store_group<true, true>(r.data, e, r.limit, raw[u]);
    }
}

// Perturb a tail tile group by group, with bounds-checked accesses (16-byte
// for whole groups of an aligned tensor, 2-byte otherwise).
template <int kThreads, int kU, int kM, bool kRows>
__device__ __forceinline__ void perturb_tail(const TileRef& r, const Streams& st) {
    const uint32_t q_hi = tile_high_word<kRows>(r);
#pragma unroll 1
    for (int u = 0; u < kU; ++u) {
        const uint64_t e = r.elem0 + uint64_t(u * kThreads + threadIdx.x) * kGroupElems;
        if (e >= r.limit) break;
        uint32_t raw[4], out[4];
        load_group<false, true>(r.data, e, r.limit, raw, r.aligned16 != 0u);
        perturb_group<kM>(raw, noise_index<kRows>(r, e), q_hi, r.tensor_id, st, out);
        store_group<false, true>(r.data, e, r.limit, out, r.aligned16 != 0u);
    }
}

// One software-pipeline step over full tiles: issue the 16-byte loads of the
// workgroup's next tile (`nxt`) into `next_buf`, read the descriptor of the
// tile after it, then perturb the current tile from `cur_buf`, so the memory
// pipe does not idle through the Philox / Box-Muller arithmetic and the
// descriptor's scalar load completes under it.  Returns true when the
// workgroup has no next tile.
//
// The loads are issued on every step, the last one reloading its own tile
// into the idle buffer (128 KB per workgroup per pass, never used), and the
// descriptor index is clamped rather than tested: the compiler's wait before
// the current tile's arithmetic is path-insensitive, and a path without loads
// after the current tile's made it wait for the next tile's loads as well.
template <int kThreads, int kU, int kM, bool kRows>
__device__ __forceinline__ bool perturb_step(const DevTile* __restrict__ tiles,
                                             const DevRows* __restrict__ rows, uint64_t& tile,
                                             uint64_t n_full, TileRef& cur, TileRef& nxt,
                                             uint32_t cur_buf[kU][4], uint32_t next_buf[kU][4],
                                             const Streams& st) {
    const uint64_t next = tile + gridDim.x;
    const bool more = next < n_full;
    __builtin_amdgcn_sched_barrier(0);
    load_tile<kThreads, kU>(more ? nxt : cur, next_buf);
    __builtin_amdgcn_sched_barrier(0);
    const uint64_t after_i = min(next + gridDim.x, n_full - 1);
    DevTile after = tiles[after_i];
    DevRows after_rows{};
    if constexpr (kRows) after_rows = rows[after_i];
    __builtin_amdgcn_sched_barrier(0);
    perturb_loaded<kThreads, kU, kM, kRows>(cur, cur_buf, st);
    keep_in_sgprs(after);
    if constexpr (kRows) keep_in_sgprs(after_rows);
    if (!more) return true;
    tile = next;
    cur = nxt;
    if constexpr (kRows) nxt = tile_ref(after, after_rows);
    else nxt = tile_ref(after);
    return false;
}

// One pass over the whole parameter list applying kM noise streams: full
// tiles first (16-byte nontemporal accesses, software-pipelined: two register
// buffers alternate, the loop unrolled twice), then tail tiles.  The first
// step is peeled off so that every step inside the loop starts with the same
// memory operations outstanding (the previous tile's stores, then the next
// tile's loads): the wait for the current tile then leaves both in flight.
//
// kRows: the launch over the tiles of strided blocks, each with its row map
// in `rows` (same index as its descriptor); otherwise `rows` is unused.
template <int kThreads, int kU, int kM, bool kRows>
__global__ __launch_bounds__(kThreads) void es_perturb_kernel(const DevTile* __restrict__ tiles,
                                                              uint64_t n_full, uint64_t n_tail,
                                                              const DevRows* __restrict__ rows,
                                                              Streams st) {
    uint64_t tile = blockIdx.x;
    if (tile < n_full) {
        TileRef cur = load_ref<kRows>(tiles, rows, tile);
        TileRef nxt = load_ref<kRows>(tiles, rows, min(tile + gridDim.x, n_full - 1));
        uint32_t a[kU][4], b[kU][4];
        load_tile<kThreads, kU>(cur, a);
        if (!perturb_step<kThreads, kU, kM, kRows>(tiles, rows, tile, n_full, cur, nxt, a, b,
                                                   st)) {
            for (;;) {
                if (perturb_step<kThreads, kU, kM, kRows>(tiles, rows, tile, n_full, cur, nxt, b,
                                                          a, st))
                    break;
                if (perturb_step<kThreads, kU, kM, kRows>(tiles, rows, tile, n_full, cur, nxt, a,
                                                          b, st))
                    break;
            }
        }
    }
    for (uint64_t tl = blockIdx.x; tl < n_tail; tl += gridDim.x)
        perturb_tail<kThreads, kU, kM, kRows>(load_ref<kRows>(tiles, rows, n_full + tl), st);
}

// A member applied from binary32 masters (es_perturb_master) with sigma > 0:
// bf16 values RNE(m + c eps) from the masters at mb + 4 e, the masters only
// read -- the arithmetic of es_perturb on the masters' values.  The perturb
// kernel's pipeline at half a tile per step: a half tile's masters (kU / 2
// slabs of 32 bytes per lane) take the registers a whole tile of bf16 takes
// there, so two half-tile buffers alternate, the next half's loads issued
// before the current half's arithmetic and each half's bf16 stores leaving
// in one burst.
//
// Within a slab (kThreads * 8 consecutive elements) lane t takes the quads
// at elements 4 t and 4 (kThreads + t): each 16-byte master load then covers
// 1 KB of consecutive masters per wave (one lane's 8 consecutive masters
// would take two loads of 16 bytes at a 32-byte stride, and streamed lines
// were fetched twice), and each 8-byte bf16 store 512 consecutive bytes.
// A quad is one Philox block: its two Box-Muller pairs are its elements.
template <int kThreads>
__device__ __forceinline__ uint64_t slab_quad(const TileRef& r, int slab, int q) {
    return r.elem0 + uint64_t(slab * kThreads) * kGroupElems +
           4 * (uint64_t(q) * kThreads + threadIdx.x);
}

template <int kThreads, int kH>
__device__ __forceinline__ void master_half_load(const TileRef& r, uintptr_t mb, int h,
                                                 float m[kH][8]) {
#pragma unroll
    for (int u = 0; u < kH; ++u)
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const uint64_t e = slab_quad<kThreads>(r, h * kH + u, q);
            const f32x4_t v = __builtin_nontemporal_load((const ES_GLOBAL f32x4_t*)(mb + 4 * e));
            m[u][4 * q] = v.x; m[u][4 * q + 1] = v.y; m[u][4 * q + 2] = v.z; m[u][4 * q + 3] = v.w;
        }
}

template <int kThreads, int kH, bool kRows>
__device__ __forceinline__ void master_half_apply(const TileRef& r, int h, float m[kH][8],
                                                  const Streams& st) {
    typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
    const uint32_t q_hi = tile_high_word<kRows>(r);
    uint32_t out[kH][4];
#pragma unroll
    for (int u = 0; u < kH; ++u)
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const uint64_t e = slab_quad<kThreads>(r, h * kH + u, q);
            const es::Words w = es::philox4x32_10(
                static_cast<uint32_t>(noise_index<kRows>(r, e) >> 2), q_hi, r.tensor_id,
                es::kDomainNoise, st.k0[0], st.k1[0]);
            float* x = &m[u][4 * q];
            float t, c, sn;
            es::scaled_pair(w.w0, w.w1, st.coef_k[0], t, c, sn);
            x[0] = __builtin_fmaf(t, c, x[0]);
            x[1] = __builtin_fmaf(t, sn, x[1]);
            es::scaled_pair(w.w2, w.w3, st.coef_k[0], t, c, sn);
            x[2] = __builtin_fmaf(t, c, x[2]);
            x[3] = __builtin_fmaf(t, sn, x[3]);
            out[u][2 * q] = es::pack_bf16x2(x[0], x[1]);
            out[u][2 * q + 1] = es::pack_bf16x2(x[2], x[3]);
        }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < kH; ++u)
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const uint64_t e = slab_quad<kThreads>(r, h * kH + u, q);
            const u32x2_t v = {out[u][2 * q], out[u][2 * q + 1]};
            __builtin_nontemporal_store(v, (ES_GLOBAL u32x2_t*)(r.data + e));
        }
}

// A tile's master base: its bf16 base times two plus the tensor's delta.
__device__ __forceinline__ uintptr_t master_base(const uint64_t* __restrict__ mdelta,
                                                 const TileRef& r, uint64_t i) {
    return mdelta[i] + 2 * reinterpret_cast<uintptr_t>(r.data);
}

// Full tiles: buffer a holds a tile's first half, b its second.  Each turn
// of the loop finishes the current tile's second half while the next tile's
// first half loads, then loads that tile's second half under its first
// half's arithmetic; the last tile's second half is done after the loop.
// Every path into the loop's head then has the same memory operations
// outstanding (the second half's loads, then the first half's stores), so
// its first wait leaves the stores in flight; the next tile's descriptor is
// read a turn ahead, as in the perturb kernel.  Tail tiles follow, group by
// group with bounds-checked accesses.
template <int kThreads, int kU, bool kRows>
__global__ __launch_bounds__(kThreads) void es_apply_master_kernel(
    const DevTile* __restrict__ tiles, uint64_t n_full, uint64_t n_tail,
    const DevRows* __restrict__ rows, Streams st, const uint64_t* __restrict__ mdelta) {
    static_assert(kU % 2 == 0, "a tile is taken in two halves");
    constexpr int kH = kU / 2;
    uint64_t tile = blockIdx.x;
    if (tile < n_full) {
        TileRef cur = load_ref<kRows>(tiles, rows, tile);
        uintptr_t cur_mb = master_base(mdelta, cur, tile);
        const uint64_t nxt_i = min(tile + gridDim.x, n_full - 1);
        TileRef nxt = load_ref<kRows>(tiles, rows, nxt_i);
        uintptr_t nxt_mb = master_base(mdelta, nxt, nxt_i);
        float a[kH][8], b[kH][8];
        master_half_load<kThreads, kH>(cur, cur_mb, 0, a);
        master_half_load<kThreads, kH>(cur, cur_mb, 1, b);
        __builtin_amdgcn_sched_barrier(0);
        master_half_apply<kThreads, kH, kRows>(cur, 0, a, st);
        while (tile + gridDim.x < n_full) {
            tile += gridDim.x;
            __builtin_amdgcn_sched_barrier(0);
            master_half_load<kThreads, kH>(nxt, nxt_mb, 0, a);
            __builtin_amdgcn_sched_barrier(0);
            const uint64_t after_i = min(tile + gridDim.x, n_full - 1);
            DevTile after = tiles[after_i];
            DevRows after_rows{};
            if constexpr (kRows) after_rows = rows[after_i];
            uint64_t after_d = mdelta[after_i];
            __builtin_amdgcn_sched_barrier(0);
            master_half_apply<kThreads, kH, kRows>(cur, 1, b, st);
            keep_in_sgprs(after);
            if constexpr (kRows) keep_in_sgprs(after_rows);
            asm volatile("" : "+s"(after_d));
            cur = nxt;
            cur_mb = nxt_mb;
            if constexpr (kRows) nxt = tile_ref(after, after_rows);
            else nxt = tile_ref(after);
            nxt_mb = after_d + 2 * reinterpret_cast<uintptr_t>(nxt.data);
            __builtin_amdgcn_sched_barrier(0);
            master_half_load<kThreads, kH>(cur, cur_mb, 1, b);
            __builtin_amdgcn_sched_barrier(0);
            master_half_apply<kThreads, kH, kRows>(cur, 0, a, st);
        }
        master_half_apply<kThreads, kH, kRows>(cur, 1, b, st);
    }
    for (uint64_t tl = blockIdx.x; tl < n_tail; tl += gridDim.x) {
        const TileRef r = load_ref<kRows>(tiles, rows, n_full + tl);
        const uintptr_t mb = master_base(mdelta, r, n_full + tl);
        const uint32_t q_hi = tile_high_word<kRows>(r);
#pragma unroll 1
        for (int u = 0; u < kU; ++u) {
            const uint64_t e = r.elem0 + uint64_t(u * kThreads + threadIdx.x) * kGroupElems;
            if (e >= r.limit) break;
            float m[8];
            load_master<false, true>(mb, e, r.limit, m, r.aligned16 != 0u);
            uint32_t w[8], out[4];
            group_words(static_cast<uint32_t>(noise_index<kRows>(r, e) >> 2), q_hi, r.tensor_id,
                        st.k0[0], st.k1[0], w);
            group_axpy(w, st.coef_k[0], m);
#pragma unroll
            for (int k = 0; k < 4; ++k) out[k] = es::pack_bf16x2(m[2 * k], m[2 * k + 1]);
            store_group<false, true>(r.data, e, r.limit, out, r.aligned16 != 0u);
        }
    }
}

// The in-place streaming ceiling of a plan (es_stream_pass): every element
// is read and written back as itself (XOR with `flip`, which the host passes
// as 0, so the compiler keeps the stores), over the same tiles and 16-byte
// nontemporal accesses as the passes above but without arithmetic and
// without software pipelining -- each workgroup loads a whole tile, then
// stores it.  On MI355X this is the fastest in-place stream measured (about
// 3 % above the same stream pipelined), so it bounds what any pass over the
// plan can reach.
template <int kThreads, int kU>
__global__ __launch_bounds__(kThreads) void es_stream_kernel(const DevTile* __restrict__ tiles,
                                                             uint64_t n_full, uint64_t n_tail,
                                                             uint32_t flip) {
    TileRef r{};
    if (blockIdx.x < n_full) r = tile_ref(tiles[blockIdx.x]);
    for (uint64_t tile = blockIdx.x; tile < n_full; tile += gridDim.x) {
        uint32_t raw[kU][4];
        load_tile<kThreads, kU>(r, raw);
        // the next tile's descriptor, read under this tile's loads
        DevTile next = tiles[min(tile + gridDim.x, n_full - 1)];
        __builtin_amdgcn_sched_barrier(0);      // all loads issued before the first wait
#pragma unroll
        for (int u = 0; u < kU; ++u)
#pragma unroll
            for (int k = 0; k < 4; ++k) raw[u][k] ^= flip;
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const uint64_t e = r.elem0 + uint64_t(u * kThreads + threadIdx.x) * kGroupElems;
            store_group<true, true>(r.data, e, r.limit, raw[u]);
        }
        keep_in_sgprs(next);
        r = tile_ref(next);
    }
    for (uint64_t tl = blockIdx.x; tl < n_tail; tl += gridDim.x) {
        const TileRef r = tile_ref(tiles[n_full + tl]);
#pragma unroll 1
        for (int u = 0; u < kU; ++u) {
            const uint64_t e = r.elem0 + uint64_t(u * kThreads + threadIdx.x) * kGroupElems;
            if (e >= r.limit) break;
            uint32_t raw[4];
            load_group<false, true>(r.data, e, r.limit, raw, r.aligned16 != 0u);
#pragma unroll
            for (int k = 0; k < 4; ++k) raw[k] ^= flip;
            store_group<false, true>(r.data, e, r.limit, raw, r.aligned16 != 0u);
        }
    }
}

// Parameter checksum (es_plan_checksum):
//   H = sum over every element of mix64(j K_J + tensor_id K_T + b K_B)  mod 2^64
// with j the element's index in its whole tensor, b its 16 bits and mix64
// the 64-bit finalizer of SplitMix64 (Steele, Lea and Flood, OOPSLA 2014).
// Addition mod 2^64 does not depend on the order of its terms, so H does not
// depend on the launch shape, and the checksums of disjoint shards of a tensor
// add up to the whole tensor's.  Read-only and VALU-bound (about 24
// instructions per element: 64-bit products and shifts on 32-bit lanes).
constexpr uint64_t kSumJ = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kSumT = 0xC2B2AE3D27D4EB4Full;
constexpr uint64_t kSumB = 0x165667B19E3779F9ull;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t x) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
    return x;
}

// The checksum terms of kN consecutive elements from whole-tensor index e,
// their values taken kBits at a time from `raw` (element k in bits
// kBits*k.. of the word array); with kChecked only elements below `limit`
// count.
template <int kN, int kBits, bool kChecked>
__device__ __forceinline__ uint64_t checksum_terms(const uint32_t* raw, uint64_t e,
                                                   uint64_t limit, uint64_t salt) {
    constexpr int kPerWord = 32 / kBits;
    constexpr uint32_t kMask = (1u << kBits) - 1u;
    uint64_t x = e * kSumJ + salt, acc = 0;
#pragma unroll
    for (int k = 0; k < kN; ++k) {
        const uint64_t b = (raw[k / kPerWord] >> (kBits * (k % kPerWord))) & kMask;
        const uint64_t f = mix64(x + b * kSumB);
        acc += (!kChecked || e + k < limit) ? f : 0ull;
        x += kSumJ;
    }
    return acc;
}

// Adds the workgroup's lane sums to *out: a lane-shuffle sum per wave, then
// one 64-bit atomic per workgroup.
template <int kThreads>
__device__ __forceinline__ void add_workgroup_sum(uint64_t acc, unsigned long long* out) {
    __shared__ uint64_t part[kThreads / 64];
    acc = wave_sum_u64(acc);
    if ((threadIdx.x & 63u) == 0u) part[threadIdx.x / 64] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t s = 0;
#pragma unroll
        for (int w = 0; w < kThreads / 64; ++w) s += part[w];
        atomicAdd(out, static_cast<unsigned long long>(s));
    }
}

// bf16 plan: full tiles with 16-byte loads and no per-element bound, then
// tail tiles bounds-checked.  With kRows (tiles of strided blocks) each
// term takes the element's whole-tensor index from the tile's row map.
template <int kThreads, int kU, bool kRows>
__global__ __launch_bounds__(kThreads) void es_checksum_kernel(const DevTile* __restrict__ tiles,
                                                               uint64_t n_full, uint64_t n_tail,
                                                               const DevRows* __restrict__ rows,
                                                               unsigned long long* __restrict__ out) {
    uint64_t acc = 0;
    for (uint64_t tile = blockIdx.x; tile < n_full; tile += gridDim.x) {
        const TileRef r = load_ref<kRows>(tiles, rows, tile);
        const uint64_t salt = uint64_t(r.tensor_id) * kSumT;
#pragma unroll 1
        for (int u = 0; u < kU; ++u) {
            const uint64_t e = r.elem0 + uint64_t(u * kThreads + threadIdx.x) * kGroupElems;
            uint32_t raw[4];
            load_group<true, true>(r.data, e, r.limit, raw);
            acc += checksum_terms<kGroupElems, 16, false>(raw, noise_index<kRows>(r, e), r.limit,
                                                          salt);
        }
    }
    for (uint64_t tl = blockIdx.x; tl < n_tail; tl += gridDim.x) {
        const TileRef r = load_ref<kRows>(tiles, rows, n_full + tl);
        const uint64_t salt = uint64_t(r.tensor_id) * kSumT;
#pragma unroll 1
        for (int u = 0; u < kU; ++u) {
            const uint64_t e = r.elem0 + uint64_t(u * kThreads + threadIdx.x) * kGroupElems;
            if (e >= r.limit) break;
            uint32_t raw[4];
            load_group<false, true>(r.data, e, r.limit, raw, r.aligned16 != 0u);
            const uint64_t n = noise_index<kRows>(r, e);
            // the bound moves with the index: n + (limit - e) for a row map
            acc += checksum_terms<kGroupElems, 16, true>(raw, n, kRows ? n + (r.limit - e) : r.limit,
                                                         salt);
        }
    }
    add_workgroup_sum<kThreads>(acc, out);
}

// *p = 0 before a checksum's atomics (a kernel, not a memset, so the call
// stays capturable into a HIP graph).
__global__ __launch_bounds__(64) void es_zero_u64_kernel(unsigned long long* __restrict__ p) {
    if (threadIdx.x == 0) *p = 0ull;
}

// HBM calibration over a caller's flat buffer (es_hbm_calibrate), with the
// perturb's workgroup and tile shape: kThreads lanes x kU 16-byte words per
// tile, each tile loaded whole and then stored, with nontemporal accesses
// (kNT, the passes' policy) or ordinary ones.  kMode 0 reads every word
// (their XOR leaves in one atomic per wave, so the loads are live), 1 writes
// every word (the pattern tile, u, lane, 0), 2 reads every word and writes it
// back (XOR with `flip`, which the host passes as 0, so the stores are kept).
template <bool kNT>
__device__ __forceinline__ u32x4_t cal_load(const ES_GLOBAL u32x4_t* a) {
    if constexpr (kNT) return __builtin_nontemporal_load(a);
    else return *a;
}
template <bool kNT>
__device__ __forceinline__ void cal_store(u32x4_t v, ES_GLOBAL u32x4_t* a) {
    if constexpr (kNT) __builtin_nontemporal_store(v, a);
    else *a = v;
}

template <int kThreads, int kU, int kMode, bool kNT>
__global__ __launch_bounds__(kThreads) void es_calibrate_kernel(u32x4_t* __restrict__ buf,
                                                                uint64_t n_tiles,
                                                                uint32_t* __restrict__ sink,
                                                                uint32_t flip) {
    uint32_t acc = 0;
    for (uint64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
        ES_GLOBAL u32x4_t* base =
            (ES_GLOBAL u32x4_t*)buf + tile * (uint64_t(kThreads) * kU) + threadIdx.x;
        u32x4_t v[kU];
        if constexpr (kMode != 1) {
#pragma unroll
            for (int u = 0; u < kU; ++u) v[u] = cal_load<kNT>(base + u * kThreads);
        }
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (kMode == 0) {
#pragma unroll
            for (int u = 0; u < kU; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
        } else {
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                if constexpr (kMode == 1) {
                    v[u] = u32x4_t{static_cast<uint32_t>(tile), uint32_t(u), threadIdx.x, 0u};
                } else {
                    v[u].x ^= flip; v[u].y ^= flip; v[u].z ^= flip; v[u].w ^= flip;
                }
                cal_store<kNT>(v[u], base + u * kThreads);
            }
        }
    }
    if constexpr (kMode == 0) {
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off, 64);
        if ((threadIdx.x & 63u) == 0u) atomicXor(sink, acc);
    }
}

// w == +-0, tested on the bit pattern so that the member loop's skip stays on
// the scalar unit (a binary32 compare would be a vector instruction).
__device__ __forceinline__ bool is_zero_weight(float w) {
    return (__float_as_uint(w) << 1) == 0u;
}

// One tile of the fused update: for each of the lane's groups in turn,
// acc = sum_d w_d eps_d (binary32, members in table order, zero weights
// skipped), theta <- round(theta + acc), store it.  Rounding is to nearest
// even, or stochastic (kSR) with the draws of one domain-1 Philox call per
// group under the rounding key.  The kernel is VALU-bound, so one group's
// registers are live at a time and the number of resident waves hides memory
// latency; full tiles also prefetch the next group while the current one is
// computed, which matters when N is small.
struct RoundKey {
    uint32_t k0, k1;
};

// The member reverted in the same pass as an update (es_restore_update): its
// entry in the distinct-seed table and coef * sqrt(2 ln 2), coef = -sign sigma.
struct RestoreArg {
    uint32_t d;
    float coef_k;
};

// The restore of one member on a group in registers, theta <- RNE(theta +
// coef eps), exactly as the perturb kernel computes it (group_axpy on the
// binary32 values, then RNE).  The member's update term is added by the
// member loop's own group_axpy from the same words, so the loop keeps one
// accumulation path (two paths merging into the accumulators cost register
// moves on every member); the Box-Muller transcendentals of this one member
// are evaluated twice.
__device__ __forceinline__ void restore_group(const uint32_t w[8], float coef_k, uint32_t raw[4]) {
    float x[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        x[2 * k] = es::bf16_lo(raw[k]);
        x[2 * k + 1] = es::bf16_hi(raw[k]);
    }
    group_axpy(w, coef_k, x);
#pragma unroll
    for (int k = 0; k < 4; ++k) raw[k] = es::pack_bf16x2(x[2 * k], x[2 * k + 1]);
}

// kRestore: one member (rst) is reverted first, in registers, and the update
// is added to the reverted values; with no live weight (add == false) the
// reverted values are stored as they are, as es_update would then leave them.
// kMaster == 1 (ES_UPDATE_MASTER): the update is added to the binary32
// masters at mb + 4 e instead (one rounding to binary32), and the bf16 values
// are rewritten as the masters rounded to nearest-even -- also with no live
// weight, when the masters are not written -- without reading them.
// kMaster == 2 (es_perturb_master): the members' terms are added to the
// masters in registers, m + sum w eps with one rounding for one member (the
// accumulation starts from m), and only the bf16 values are written.
template <int kThreads, int kU, bool kFast, bool kNT, bool kSR, bool kRows, bool kRestore,
          int kMaster>
__device__ __forceinline__ void update_tile(const TileRef& r, const Member* __restrict__ members,
                                            uint32_t n_distinct, RoundKey rk, RestoreArg rst,
                                            bool add, uintptr_t mb) {
    constexpr int kIn = kMaster != 0 ? 8 : 4;            // words of a group's input
    const uint32_t q_hi = tile_high_word<kRows>(r);
    const uint32_t g_hi = q_hi >> 1;                     // index >> 35
    const uint64_t e0 = r.elem0 + uint64_t(threadIdx.x) * kGroupElems;
    uint32_t next[kIn];
    auto load_in = [&](auto fast, uint64_t e, uint32_t in[kIn]) {
        constexpr bool kF = decltype(fast)::value;
        if constexpr (kMaster != 0) {
            float m[8];
            load_master<kF, kNT>(mb, e, r.limit, m, r.aligned16 != 0u);
#pragma unroll
            for (int k = 0; k < 8; ++k) in[k] = __builtin_bit_cast(uint32_t, m[k]);
        } else {
            load_group<kF, kNT>(r.data, e, r.limit, in, r.aligned16 != 0u);
        }
    };
    if constexpr (kFast) load_in(std::true_type{}, e0, next);
#pragma unroll 1
    for (int u = 0; u < kU; ++u) {
        const uint64_t e = e0 + uint64_t(u) * kThreads * kGroupElems;
        if (!kFast && e >= r.limit) break;
        uint32_t raw[kIn];
        if constexpr (kFast) {
#pragma unroll
            for (int k = 0; k < kIn; ++k) raw[k] = next[k];
            if (u + 1 < kU) load_in(std::true_type{}, e + uint64_t(kThreads) * kGroupElems, next);
        } else {
            load_in(std::false_type{}, e, raw);
        }
        const uint64_t n = noise_index<kRows>(r, e);
        const uint32_t q_lo = static_cast<uint32_t>(n >> 2);
        float acc[8];
#pragma unroll
        for (int k = 0; k < 8; ++k)
            acc[k] = kMaster == 2 ? __builtin_bit_cast(float, raw[k]) : 0.0f;
        for (uint32_t d = 0; d < n_distinct; ++d) {
            const Member m = members[d];
            const bool live = !is_zero_weight(m.w_k);
            if constexpr (kRestore) {
                if (!live && d != rst.d) continue;
            } else {
                if (!live) continue;
            }
            uint32_t w[8];
            group_words(q_lo, q_hi, r.tensor_id, m.k0, m.k1, w);
            if constexpr (kRestore) {
                if (d == rst.d) restore_group(w, rst.coef_k, raw);
                if (!live) continue;
            }
            group_axpy(w, m.w_k, acc);
        }
        uint32_t out[4];
        if constexpr (kMaster == 2) {
#pragma unroll
            for (int k = 0; k < 4; ++k) out[k] = es::pack_bf16x2(acc[2 * k], acc[2 * k + 1]);
        } else if constexpr (kMaster == 1) {
            float m[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) m[k] = __builtin_bit_cast(float, raw[k]);
            if (add) {
#pragma unroll
                for (int k = 0; k < 8; ++k) m[k] += acc[k];
                store_master<kFast, kNT>(mb, e, r.limit, m, r.aligned16 != 0u);
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) out[k] = es::pack_bf16x2(m[2 * k], m[2 * k + 1]);
        } else if (kRestore && !add) {
#pragma unroll
            for (int k = 0; k < 4; ++k) out[k] = raw[k];
        } else if constexpr (kSR) {
            const es::Words d = es::philox4x32_10(static_cast<uint32_t>(n >> 3), g_hi, r.tensor_id,
                                                  es::kDomainRounding, rk.k0, rk.k1);
            const uint32_t draws[4] = {d.w0, d.w1, d.w2, d.w3};
#pragma unroll
            for (int k = 0; k < 4; ++k)
                out[k] = es::pack_bf16x2_sr(es::bf16_lo(raw[k]) + acc[2 * k],
                                            es::bf16_hi(raw[k]) + acc[2 * k + 1], draws[k]);
        } else {
#pragma unroll
            for (int k = 0; k < 4; ++k)
                out[k] = es::pack_bf16x2(es::bf16_lo(raw[k]) + acc[2 * k],
                                         es::bf16_hi(raw[k]) + acc[2 * k + 1]);
        }
        store_group<kFast, kNT>(r.data, e, r.limit, out, r.aligned16 != 0u);
    }
}

// Fused update over the whole parameter list (member table and header
// written by es_prepare_kernel): full tiles, then tail tiles; with kRows the
// tiles of strided blocks, through their row maps; with kRestore the member
// rst reverted in the same pass.
template <int kThreads, int kU, bool kNT, bool kSR, bool kRows, bool kRestore, int kMaster>
__global__ __launch_bounds__(kThreads) void es_update_kernel(const DevTile* __restrict__ tiles,
                                                             uint64_t n_full, uint64_t n_tail,
                                                             const DevRows* __restrict__ rows,
                                                             const Member* __restrict__ members,
                                                             const UpdateHeader* __restrict__ hdr,
                                                             RoundKey rk, RestoreArg rst,
                                                             const uint64_t* __restrict__ mdelta) {
    const bool add = hdr->n_live != 0u;
    if (!kRestore && kMaster == 0 && !add) return;   // nothing to add: theta is not written
    const uint32_t n_distinct = hdr->n_distinct;
    // a tile's master base: its bf16 base times two plus the tensor's delta
    auto mbase = [&](const TileRef& r, uint64_t i) -> uintptr_t {
        if constexpr (kMaster != 0) return mdelta[i] + 2 * reinterpret_cast<uintptr_t>(r.data);
        else return 0;
    };
    for (uint64_t tile = blockIdx.x; tile < n_full; tile += gridDim.x) {
        const TileRef r = load_ref<kRows>(tiles, rows, tile);
        update_tile<kThreads, kU, true, kNT, kSR, kRows, kRestore, kMaster>(
            r, members, n_distinct, rk, rst, add, mbase(r, tile));
    }
    for (uint64_t tile = blockIdx.x; tile < n_tail; tile += gridDim.x) {
        const TileRef r = load_ref<kRows>(tiles, rows, n_full + tile);
        update_tile<kThreads, kU, false, kNT, kSR, kRows, kRestore, kMaster>(
            r, members, n_distinct, rk, rst, add, mbase(r, n_full + tile));
    }
}

// The scratch of es_update_noalloc: one update's staged member tables, merged
// weights and header (the layout of a plan's scratch), in a fixed device
// array instead of memory allocated with a plan.  Each device holds its own
// copy until the process ends; host code reaches it only through the address
// hipGetSymbolAddress returns for the current device.
__device__ __align__(256) uint8_t scratch[kScratchBytes];

// Copy up to 1 KB of host-packed words (passed as kernel arguments) into
// device scratch: how es_update hands its member tables to the device
// without a host-side staging buffer or synchronisation.
__global__ __launch_bounds__(kAuxBlock) void es_stage_kernel(uint32_t* __restrict__ dst,
                                                          uint32_t n_words, StageChunk chunk) {
    for (uint32_t i = threadIdx.x; i < n_words; i += blockDim.x) dst[i] = chunk.words[i];
}

// Wave-wide reductions (one wavefront of 64 lanes).
__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
    return x;
}
__device__ __forceinline__ float wave_min(float x) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x = fminf(x, __shfl_xor(x, off, 64));
    return x;
}
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
    return x;
}

// Population z-score of n rewards by one wavefront, fp64, into LDS z[].
// Returns the status (1 if any reward is not finite; then z = 0).  All
// rewards equal gives z = 0 exactly.
__device__ int wave_zscore(const float* __restrict__ r, uint32_t n, double eps, double* z) {
    const uint32_t lane = threadIdx.x;
    double s = 0.0;
    float lo = INFINITY, hi = -INFINITY;
    int bad = 0;
    for (uint32_t i = lane; i < n; i += 64) {
        const float x = r[i];
        bad |= !isfinite(x);
        s += static_cast<double>(x);
        lo = fminf(lo, x);
        hi = fmaxf(hi, x);
    }
    bad = __any(bad);
    if (bad) {
        for (uint32_t i = lane; i < n; i += 64) z[i] = 0.0;
        return 1;
    }
    lo = wave_min(lo);
    hi = wave_max(hi);
    if (lo == hi) {
        for (uint32_t i = lane; i < n; i += 64) z[i] = 0.0;
        return 0;
    }
    const double mu = wave_sum(s) / static_cast<double>(n);
    double q = 0.0;
    for (uint32_t i = lane; i < n; i += 64) {
        const double d = static_cast<double>(r[i]) - mu;
        q += d * d;
    }
    const double sd = sqrt(wave_sum(q) / static_cast<double>(n));
    for (uint32_t i = lane; i < n; i += 64) z[i] = (static_cast<double>(r[i]) - mu) / (sd + eps);
    return 0;
}

__global__ __launch_bounds__(64) void es_zscore_kernel(const float* __restrict__ r, uint32_t n,
                                                       double eps, float* __restrict__ z_out,
                                                       int32_t* __restrict__ status_out) {
    __shared__ double z[ES_MAX_MEMBERS];
    const int status = wave_zscore(r, n, eps, z);
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < n; i += 64) z_out[i] = static_cast<float>(z[i]);
    if (status_out != nullptr && threadIdx.x == 0) *status_out = status;
}

// z-score (or rewards as weights), then one merged weight per distinct seed:
// w_d = sum over its members (in member order) of c * sign * zhat, fp64,
// stored as binary32 with the seed's key for es_update_kernel.
__global__ __launch_bounds__(64) void es_prepare_kernel(
    const float* __restrict__ r, uint32_t n, double eps, uint32_t flags, double c,
    const MemberIn* __restrict__ min, const DistinctIn* __restrict__ din, uint32_t n_distinct,
    Member* __restrict__ out, UpdateHeader* __restrict__ hdr, float* __restrict__ z_out,
    int32_t* __restrict__ status_out) {
    __shared__ double z[ES_MAX_MEMBERS];
    const uint32_t lane = threadIdx.x;
    int status;
    if (flags & ES_REWARDS_ARE_WEIGHTS) {
        int bad = 0;
        for (uint32_t i = lane; i < n; i += 64) {
            const float x = r[i];
            bad |= !isfinite(x);
            z[i] = static_cast<double>(x);
        }
        status = __any(bad) ? 1 : 0;
    } else {
        status = wave_zscore(r, n, eps, z);
    }
    __syncthreads();
    if (z_out != nullptr)
        for (uint32_t i = lane; i < n; i += 64) z_out[i] = static_cast<float>(status ? 0.0 : z[i]);
    uint32_t live = 0;
    for (uint32_t d = lane; d < n_distinct; d += 64) {
        const DistinctIn di = din[d];
        double w = 0.0;
        for (uint32_t m = di.first; m < di.first + di.count; ++m)
            w += c * static_cast<double>(min[m].sign) * z[min[m].reward_index];
        const float wf = status ? 0.0f : static_cast<float>(w * kSqrt2Ln2Double);
        out[d] = Member{di.k0, di.k1, wf, 0u};
        live += (wf != 0.0f) ? 1u : 0u;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) live += __shfl_xor(live, off, 64);
    if (lane == 0) {
        *hdr = UpdateHeader{n_distinct, live, status, 0u};
        if (status_out != nullptr) *status_out = status;
    }
}

__global__ __launch_bounds__(kAuxBlock) void es_philox_words_kernel(uint32_t k0, uint32_t k1,
                                                                 uint32_t tensor_id, uint32_t domain,
                                                                 uint64_t quad0, uint64_t n_quads,
                                                                 uint4* __restrict__ out) {
    const uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n_quads) return;
    const uint64_t q = quad0 + i;
    const es::Words w = es::philox4x32_10(static_cast<uint32_t>(q), static_cast<uint32_t>(q >> 32),
                                          tensor_id, domain, k0, k1);
    out[i] = make_uint4(w.w0, w.w1, w.w2, w.w3);
}

__global__ __launch_bounds__(kAuxBlock) void es_normals_kernel(uint32_t k0, uint32_t k1,
                                                            uint32_t tensor_id, uint64_t elem0,
                                                            uint64_t n, float* __restrict__ out) {
    const uint64_t q = (elem0 >> 2) + uint64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (4 * q >= elem0 + n) return;
    float e[4];
    es::quad_normals(static_cast<uint32_t>(q), static_cast<uint32_t>(q >> 32), tensor_id, k0, k1, e);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint64_t j = 4 * q + k;
        if (j >= elem0 && j < elem0 + n) out[j - elem0] = e[k];
    }
}

using PerturbKernel = void (*)(const DevTile*, uint64_t, uint64_t, const DevRows*, Streams);
using UpdateKernel = void (*)(const DevTile*, uint64_t, uint64_t, const DevRows*, const Member*,
                              const UpdateHeader*, RoundKey, RestoreArg, const uint64_t*);

// Tile shapes instantiated: T lanes per workgroup x U groups per lane.
#define ES_TILE_SHAPES(X) X(256, 4) X(256, 8) X(512, 4) X(512, 8) X(1024, 4) X(1024, 8)

template <int kM, bool kRows>
PerturbKernel perturb_kernel_for(int threads, int groups) {
#define ES_CASE(T, U) if (threads == T && groups == U) return es_perturb_kernel<T, U, kM, kRows>;
    ES_TILE_SHAPES(ES_CASE)
#undef ES_CASE
    return nullptr;
}

using StreamKernel = void (*)(const DevTile*, uint64_t, uint64_t, uint32_t);

StreamKernel stream_kernel(int threads, int groups) {
#define ES_CASE(T, U) if (threads == T && groups == U) return es_stream_kernel<T, U>;
    ES_TILE_SHAPES(ES_CASE)
#undef ES_CASE
    return nullptr;
}

using ChecksumKernel = void (*)(const DevTile*, uint64_t, uint64_t, const DevRows*,
                                unsigned long long*);

ChecksumKernel checksum_kernel(int threads, int groups, bool rows) {
#define ES_CASE(T, U)                                                                     \
    if (threads == T && groups == U)                                                      \
        return rows ? es_checksum_kernel<T, U, true> : es_checksum_kernel<T, U, false>;
    ES_TILE_SHAPES(ES_CASE)
#undef ES_CASE
    return nullptr;
}

// streams: 1 (perturb / restore), 2 (swap, two keys), 3 (swap, one key);
// rows: the launch over strided blocks' tiles.
PerturbKernel perturb_kernel(int streams, int threads, int groups, bool rows) {
    switch (streams * 2 + (rows ? 1 : 0)) {
        case 2: return perturb_kernel_for<1, false>(threads, groups);
        case 3: return perturb_kernel_for<1, true>(threads, groups);
        case 4: return perturb_kernel_for<2, false>(threads, groups);
        case 5: return perturb_kernel_for<2, true>(threads, groups);
        case 6: return perturb_kernel_for<3, false>(threads, groups);
        case 7: return perturb_kernel_for<3, true>(threads, groups);
        default: return nullptr;
    }
}

template <bool kRestore>
UpdateKernel update_kernel_for(int threads, int groups, bool stochastic, bool rows) {
#define ES_CASE(T, U)                                                                        \
    if (threads == T && groups == U) {                                                       \
        if (rows)                                                                            \
            return stochastic ? es_update_kernel<T, U, true, true, true, kRestore, 0>    \
                              : es_update_kernel<T, U, true, false, true, kRestore, 0>;  \
        return stochastic ? es_update_kernel<T, U, true, true, false, kRestore, 0>       \
                          : es_update_kernel<T, U, true, false, false, kRestore, 0>;     \
    }
    ES_TILE_SHAPES(ES_CASE)
#undef ES_CASE
    return nullptr;
}

// The update into binary32 masters (mode 1) and the application of members
// from the masters (mode 2), both rewriting the bf16 values.
template <int kMode>
UpdateKernel master_kernel_for(int threads, int groups, bool rows) {
#define ES_CASE(T, U)                                                                   \
    if (threads == T && groups == U)                                                    \
        return rows ? es_update_kernel<T, U, true, false, true, false, kMode>           \
                    : es_update_kernel<T, U, true, false, false, false, kMode>;
    ES_TILE_SHAPES(ES_CASE)
#undef ES_CASE
    return nullptr;
}

using ApplyMasterKernel = void (*)(const DevTile*, uint64_t, uint64_t, const DevRows*, Streams,
                                   const uint64_t*);

ApplyMasterKernel apply_master_kernel(int threads, int groups, bool rows) {
#define ES_CASE(T, U)                                                                   \
    if (threads == T && groups == U)                                                    \
        return rows ? es_apply_master_kernel<T, U, true> : es_apply_master_kernel<T, U, false>;
    ES_TILE_SHAPES(ES_CASE)
#undef ES_CASE
    return nullptr;
}

UpdateKernel update_master_kernel(int threads, int groups, bool rows, bool apply = false) {
    return apply ? master_kernel_for<2>(threads, groups, rows)
                 : master_kernel_for<1>(threads, groups, rows);
}

// restore: the update with one member reverted in the same pass.
UpdateKernel update_kernel(int threads, int groups, bool stochastic, bool rows,
                           bool restore = false) {
    return restore ? update_kernel_for<true>(threads, groups, stochastic, rows)
                   : update_kernel_for<false>(threads, groups, stochastic, rows);
}

// ---- quantized path: int8 and E4M3 codes (helpers in es_quant.hpp, es_fp8.hpp) ----

// Kernel arguments of one quantized pass: the key of the update's rounding
// draws, and for perturb / restore the single member inline (for a swap, m is
// the member applied and m_from the member reverted before it).
struct QPass {
    uint32_t dk0, dk1;
    uint32_t pad0, pad1;
    Member m;
    Member m_from;
};

// Perturb / restore of one 16-code group (n: the whole-tensor index of its
// first code): per quad of codes one noise call, whose words give the four
// normals and the four rounding draws.  The scale's reciprocal is folded into
// the pair's radius factor, and d + f is one FMA.
template <bool kNegate>
__device__ __forceinline__ void qperturb_group(const uint32_t raw[4], uint32_t n,
                                               uint32_t tensor_id, const Member& m, float inv0,
                                               float inv1, uint32_t out[4]) {
    const uint32_t q = n >> 2;                  // multiple of 4: q + 3 does not carry
    // an invalid scale has inv = 0: its step is 0 and its codes clamp to
    // [-128, 127], i.e. they are left as they are
    const float wk_inv[2] = {m.w_k * inv0, m.w_k * inv1};
    const int32_t lo[2] = {inv0 != 0.0f ? -127 : -128, inv1 != 0.0f ? -127 : -128};
    const uint32_t one_plus = esq::one_plus_half_step_vgpr();
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const es::Words w = es::philox4x32_10(q + c, 0u, tensor_id, es::kDomainNoise, m.k0, m.k1);
        const uint32_t ws[4] = {w.w0, w.w1, w.w2, w.w3};
        int32_t code[4];
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            float t, cs, sn;
            es::scaled_pair(ws[2 * p], ws[2 * p + 1], wk_inv[c >> 1], t, cs, sn);
            const float trig[2] = {cs, sn};
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int i = 2 * p + h;
                const int32_t qc = static_cast<int8_t>(raw[c] >> (8 * i));
                const float v = __builtin_fmaf(t, trig[h], esq::spare_one_plus(ws[i], one_plus));
                code[i] = esq::qstep9<kNegate>(qc, v, lo[c >> 1]);
            }
        }
        out[c] = esq::pack_codes(code[0], code[1], code[2], code[3]);
    }
}

// Code formats of a quantized plan.
constexpr int kFmtInt8 = 0;
constexpr int kFmtE4M3 = 1;

// fp8 perturb / restore of one 16-code group (n as above): per quad of codes one noise
// call, whose words give the four normals and the four spare draws.  The
// scale's reciprocal is folded into the pair's radius factor; x = v -+ d is
// one fused multiply-add, and the restore rounds with the complementary
// rule (operand ~U for U), so it undoes the perturbation inside a binade.
template <bool kNegate>
__device__ __forceinline__ void f8perturb_group(const uint32_t raw[4], uint32_t n,
                                                uint32_t tensor_id, const Member& m, float inv0,
                                                float inv1, uint32_t out[4]) {
    const uint32_t q = n >> 2;                  // multiple of 4: q + 3 does not carry
    const float wk_inv[2] = {m.w_k * inv0, m.w_k * inv1};
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const es::Words w = es::philox4x32_10(q + c, 0u, tensor_id, es::kDomainNoise, m.k0, m.k1);
        const uint32_t ws[4] = {w.w0, w.w1, w.w2, w.w3};
        float v[4], x[4];
        uint32_t a[4];
        esf::decode4(raw[c], v);
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            float t, cs, sn;
            es::scaled_pair(ws[2 * p], ws[2 * p + 1], wk_inv[c >> 1], t, cs, sn);
            const float trig[2] = {cs, sn};
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int i = 2 * p + h;
                const uint32_t u = esf::draw9_fixed(ws[i]);
                x[i] = __builtin_fmaf(kNegate ? -t : t, trig[h], v[i]);
                a[i] = kNegate ? ~u : u;
            }
        }
        out[c] = esf::round4(x, a);
    }
}

// Perturb (kNegate false) or restore of one 16-code group in the plan's
// format, codes with an invalid scale or a not-a-number code left as they are.
template <bool kNegate, int kFmt>
__device__ __forceinline__ void qmember_group(const uint32_t raw[4], uint32_t n,
                                              uint32_t tensor_id, const Member& m, float inv0,
                                              float inv1, uint32_t out[4]) {
    if constexpr (kFmt == kFmtE4M3) {
        f8perturb_group<kNegate>(raw, n, tensor_id, m, inv0, inv1, out);
        esf::keep_special(raw, inv0, inv1, out);
    } else {
        qperturb_group<kNegate>(raw, n, tensor_id, m, inv0, inv1, out);
    }
}

// One tile of a quantized pass (int8 or E4M3 codes, kFmt): for each of the
// lane's 16-code groups in turn, the step in scale units (binary32) and the
// stochastically rounded, clamped code.  e indexes the codes and scales at hand; n, the whole-tensor index
// of code e, selects the noise and the rounding draws.
// kSwap: the member ps.m_from reverted and ps.m applied in registers, the
// codes of the two separate passes.
template <int kThreads, int kU, bool kFast, bool kTable, bool kNegate, int kFmt, bool kSwap>
__device__ __forceinline__ void qtile(const esq::QTileRef& r, const Member* __restrict__ members,
                                      uint32_t n_members, const QPass& ps) {
    const uint32_t e0 = r.elem0 + threadIdx.x * esq::kQGroup;
#pragma unroll 1
    for (int u = 0; u < kU; ++u) {
        const uint32_t e = e0 + uint32_t(u) * kThreads * esq::kQGroup;
        if (!kFast && e >= r.numel) break;
        const uint32_t n = esq::qnoise_index(r, e);
        uint32_t raw[4];
        esq::qload<kFast>(r.data, e, r.numel, raw, r.aligned16 != 0u);
        float inv0, inv1;
        esq::group_inv_scales(r, e, inv0, inv1);
        uint32_t out[4];
        if constexpr (kSwap) {
            uint32_t mid[4];
            qmember_group<true, kFmt>(raw, n, r.tensor_id, ps.m_from, inv0, inv1, mid);
            qmember_group<false, kFmt>(mid, n, r.tensor_id, ps.m, inv0, inv1, out);
        } else if constexpr (!kTable) {
            qmember_group<kNegate, kFmt>(raw, n, r.tensor_id, ps.m, inv0, inv1, out);
        } else {
            float acc[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[i] = 0.0f;
            for (uint32_t d = 0; d < n_members; ++d) {
                const Member m = members[d];
                if (is_zero_weight(m.w_k)) continue;
                esq::qgroup_axpy(n, r.tensor_id, m.k0, m.k1, m.w_k, acc);
            }
            const es::Words da =
                es::philox4x32_10(n >> 3, 0u, r.tensor_id, es::kDomainRounding, ps.dk0, ps.dk1);
            const es::Words db = es::philox4x32_10((n >> 3) + 1u, 0u, r.tensor_id,
                                                   es::kDomainRounding, ps.dk0, ps.dk1);
            const uint32_t dw[8] = {da.w0, da.w1, da.w2, da.w3, db.w0, db.w1, db.w2, db.w3};
            if constexpr (kFmt == kFmtE4M3) {
                // x = v + acc / s (one fused multiply-add), rounded onto the
                // grid with the threshold 1 - r 2^-16 (operand r 2^16)
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    float v[4], x[4];
                    uint32_t a[4];
                    esf::decode4(raw[k], v);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int c = 4 * k + i;
                        const uint32_t d = dw[c >> 1];
                        a[i] = (c & 1) ? (d & 0xFFFF0000u) : (d << 16);
                        x[i] = __builtin_fmaf(acc[c], c < 8 ? inv0 : inv1, v[i]);
                    }
                    out[k] = esf::round4(x, a);
                }
                esf::keep_special(raw, inv0, inv1, out);
            } else {
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    uint32_t w = 0;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int c = 4 * k + i;
                        const float inv = c < 8 ? inv0 : inv1;
                        const int32_t q = static_cast<int8_t>(raw[k] >> (8 * i));
                        const uint32_t draw = (dw[c >> 1] >> (16 * (c & 1))) & 0xFFFFu;
                        const int32_t v =
                            inv != 0.0f ? esq::qstep<false>(q, acc[c] * inv, draw) : q;
                        w |= (static_cast<uint32_t>(v) & 0xFFu) << (8 * i);
                    }
                    out[k] = w;
                }
            }
        }
        esq::qstore<kFast>(r.data, e, r.numel, out, r.aligned16 != 0u);
    }
}

// A pass over the whole quantized parameter list: perturb / restore (one
// inline member, draws from its own noise words), swap (two inline members)
// or the update (member table and header written by es_prepare_kernel, draws
// of domain 1 under the rounding seed).
template <int kThreads, int kU, bool kTable, bool kNegate, int kFmt, bool kSwap>
__global__ __launch_bounds__(kThreads) void es_qpass_kernel(const esq::DevQTensor* __restrict__ tab,
                                                            uint64_t n_full, uint64_t n_tail,
                                                            const Member* __restrict__ members,
                                                            const UpdateHeader* __restrict__ hdr,
                                                            QPass ps) {
    constexpr uint32_t kTileElems = uint32_t(kThreads) * kU * esq::kQGroup;
    uint32_t n_members = 1;
    if constexpr (kTable) {
        if (hdr->n_live == 0u) return;      // nothing to add: codes are not written
        n_members = hdr->n_distinct;
    }
    uint32_t t = 0;
    for (uint64_t tile = blockIdx.x; tile < n_full; tile += gridDim.x)
        qtile<kThreads, kU, true, kTable, kNegate, kFmt, kSwap>(
            esq::qlocate_full<kTileElems>(tab, t, tile), members, n_members, ps);
    t = 0;
    for (uint64_t tile = blockIdx.x; tile < n_tail; tile += gridDim.x)
        qtile<kThreads, kU, false, kTable, kNegate, kFmt, kSwap>(
            esq::qlocate_tail<kTileElems>(tab, t, tile), members, n_members, ps);
}

using QPassKernel = void (*)(const esq::DevQTensor*, uint64_t, uint64_t, const Member*,
                             const UpdateHeader*, QPass);

enum class QKind { kPerturb, kRestore, kUpdate, kSwap };

template <int kFmt>
QPassKernel qpass_kernel_for(int threads, int groups, QKind kind) {
#define ES_CASE(T, U)                                                                      \
    if (threads == T && groups == U) {                                                     \
        switch (kind) {                                                                    \
            case QKind::kPerturb: return es_qpass_kernel<T, U, false, false, kFmt, false>; \
            case QKind::kRestore: return es_qpass_kernel<T, U, false, true, kFmt, false>;  \
            case QKind::kUpdate: return es_qpass_kernel<T, U, true, false, kFmt, false>;   \
            case QKind::kSwap: return es_qpass_kernel<T, U, false, false, kFmt, true>;     \
        }                                                                                  \
    }
    ES_TILE_SHAPES(ES_CASE)
#undef ES_CASE
    return nullptr;
}

QPassKernel qpass_kernel(int threads, int groups, QKind kind, int format) {
    return format == kFmtE4M3 ? qpass_kernel_for<kFmtE4M3>(threads, groups, kind)
                              : qpass_kernel_for<kFmtInt8>(threads, groups, kind);
}

// Quantized plan: the same sum with b the code's 8 bits and j the element's
// whole-tensor index (qnoise_index; a 16-code group's indices are
// consecutive).
template <int kThreads, int kU>
__global__ __launch_bounds__(kThreads) void es_qchecksum_kernel(
    const esq::DevQTensor* __restrict__ tab, uint64_t n_full, uint64_t n_tail,
    unsigned long long* __restrict__ out) {
    constexpr uint32_t kTileElems = uint32_t(kThreads) * kU * esq::kQGroup;
    uint64_t acc = 0;
    uint32_t t = 0;
    for (uint64_t tile = blockIdx.x; tile < n_full; tile += gridDim.x) {
        const esq::QTileRef r = esq::qlocate_full<kTileElems>(tab, t, tile);
        const uint64_t salt = uint64_t(r.tensor_id) * kSumT;
#pragma unroll 1
        for (int u = 0; u < kU; ++u) {
            const uint32_t e = r.elem0 + (uint32_t(u) * kThreads + threadIdx.x) * esq::kQGroup;
            uint32_t raw[4];
            esq::qload<true>(r.data, e, r.numel, raw);
            acc += checksum_terms<esq::kQGroup, 8, false>(raw, esq::qnoise_index(r, e), 0, salt);
        }
    }
    t = 0;
    for (uint64_t tile = blockIdx.x; tile < n_tail; tile += gridDim.x) {
        const esq::QTileRef r = esq::qlocate_tail<kTileElems>(tab, t, tile);
        const uint64_t salt = uint64_t(r.tensor_id) * kSumT;
#pragma unroll 1
        for (int u = 0; u < kU; ++u) {
            const uint32_t e = r.elem0 + (uint32_t(u) * kThreads + threadIdx.x) * esq::kQGroup;
            if (e >= r.numel) break;
            uint32_t raw[4];
            esq::qload<false>(r.data, e, r.numel, raw, r.aligned16 != 0u);
            const uint32_t n = esq::qnoise_index(r, e);
            acc += checksum_terms<esq::kQGroup, 8, true>(raw, n, uint64_t(n) + (r.numel - e),
                                                         salt);
        }
    }
    add_workgroup_sum<kThreads>(acc, out);
}

using QChecksumKernel = void (*)(const esq::DevQTensor*, uint64_t, uint64_t, unsigned long long*);

QChecksumKernel qchecksum_kernel(int threads, int groups) {
#define ES_CASE(T, U) if (threads == T && groups == U) return es_qchecksum_kernel<T, U>;
    ES_TILE_SHAPES(ES_CASE)
#undef ES_CASE
    return nullptr;
}

}  // namespace

// ------------------------------------------------------------------------
// Host side
// ------------------------------------------------------------------------

struct es_plan {
    int device = -1;
    uint32_t n_tensors = 0;
    uint64_t numel = 0;
    uint64_t n_full = 0;            // full tiles (16-byte path)
    uint64_t n_tail = 0;            // tail tiles (bounds-checked path)
    uint64_t n_rfull = 0;           // full and tail tiles of strided blocks, after the
    uint64_t n_rtail = 0;           //   others, each with a row map
    uint32_t grid_perturb = 0;      // workgroups of the perturb / restore launch
    uint32_t grid_update = 0;       // workgroups of the update launch
    uint32_t grid_perturb_rows = 0; // the same for the strided blocks' launch
    uint32_t grid_update_rows = 0;
    int threads = kDefaultThreads;  // lanes per workgroup of the tile kernels
    int groups = kDefaultGroups;    // 8-element groups per lane per tile
    uint64_t tile_elems = 0;        // threads * groups * 8
    DevTile* d_tiles = nullptr;     // n_full full-tile then n_tail tail-tile descriptors, then
                                    //   n_rfull + n_rtail of strided blocks
    DevRows* d_rows = nullptr;      // their row maps (same allocation, after the descriptors)
    uint8_t* d_scratch = nullptr;   // kScratchBytes
    // each tensor's or block's bf16 data and element count, in plan order
    std::vector<std::pair<uintptr_t, uint64_t>> owners;
    // binary32 masters (es_plan_set_master): per tile, the delta D with
    // master address = D + 2 * bf16 address (its tensor's master minus twice
    // its bf16 data pointer, mod 2^64); null when none are attached
    uint64_t* d_master = nullptr;
};

struct es_qplan {
    int device = -1;
    uint32_t n_tensors = 0;
    uint64_t numel = 0;
    uint64_t n_full = 0;
    uint64_t n_tail = 0;
    uint32_t grid = 0;              // workgroups of every quantized pass
    int threads = kDefaultThreads;
    int groups = kDefaultQGroups;   // 16-code groups per lane per tile
    int format = kFmtInt8;          // ES_QFORMAT_INT8 or ES_QFORMAT_E4M3 (one per plan)
    esq::DevQTensor* d_tab = nullptr;
    uint8_t* d_scratch = nullptr;   // kScratchBytes, as the bf16 plan's
};

namespace {

// Integer from the environment within [lo, hi], else the default.
int env_int(const char* name, int dflt, int lo, int hi) {
    const char* v = std::getenv(name);
    if (v == nullptr) return dflt;
    const int x = std::atoi(v);
    return (x >= lo && x <= hi) ? x : dflt;
}

int check_device(const es_plan_t* p) {
    int dev = -1;
    const hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != p->device)
        return fail(ES_ERR_DEVICE, "current device " + std::to_string(dev) +
                                       " differs from the plan's device " +
                                       std::to_string(p->device));
    return ES_OK;
}

// The launches of a pass over a plan: one over the tiles of tensors and
// contiguous blocks, and one over the tiles of strided blocks with their
// row maps; a part with no tiles is left out.
struct Segment {
    const DevTile* tiles;
    uint64_t n_full, n_tail;
    const DevRows* rows;            // null for the first part
    uint32_t grid_perturb, grid_update;
};

int plan_segments(const es_plan_t* p, Segment seg[2]) {
    int n = 0;
    if (p->n_full + p->n_tail > 0)
        seg[n++] = Segment{p->d_tiles, p->n_full, p->n_tail, nullptr, p->grid_perturb,
                           p->grid_update};
    if (p->n_rfull + p->n_rtail > 0)
        seg[n++] = Segment{p->d_tiles + p->n_full + p->n_tail, p->n_rfull, p->n_rtail, p->d_rows,
                           p->grid_perturb_rows, p->grid_update_rows};
    return n;
}

// One pass of the perturb kernel: streams = 1 (seed[0], coef[0]), 2 (two
// keys) or 3 (both coefficients on seed[0]).
int launch_streams(es_plan_t* p, int streams, const uint64_t* seed, const double* coef,
                   hipStream_t s) {
    Streams st = {};
    const int terms = streams == 1 ? 1 : 2;
    for (int m = 0; m < terms; ++m) {
        const uint64_t sd = streams == 3 ? seed[0] : seed[m];
        st.k0[m] = static_cast<uint32_t>(sd);
        st.k1[m] = static_cast<uint32_t>(sd >> 32);
        st.coef_k[m] = static_cast<float>(coef[m] * kSqrt2Ln2Double);
    }
    Segment seg[2];
    const int n_seg = plan_segments(p, seg);
    for (int k = 0; k < n_seg; ++k) {
        const Segment& g = seg[k];
        const PerturbKernel kernel = perturb_kernel(streams, p->threads, p->groups, g.rows != nullptr);
        hipLaunchKernelGGL(kernel, dim3(g.grid_perturb), dim3(p->threads), 0, s, g.tiles, g.n_full,
                           g.n_tail, g.rows, st);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(e, "es_perturb_kernel launch");
    }
    return ES_OK;
}

int perturb_impl(es_plan_t* p, uint64_t seed, int32_t sign, float sigma, es_stream_t stream,
                 const char* name) {
    if (p == nullptr) return fail(ES_ERR_INVALID_ARG, std::string(name) + ": null plan");
    if (sign != 1 && sign != -1)
        return fail(ES_ERR_INVALID_ARG, std::string(name) + ": sign must be +1 or -1");
    if (!std::isfinite(sigma) || sigma < 0.0f)
        return fail(ES_ERR_INVALID_ARG, std::string(name) + ": sigma must be finite and >= 0");
    if (sigma == 0.0f) return ES_OK;
    const int rc = check_device(p);
    if (rc != ES_OK) return rc;
    const double coef = sign > 0 ? double(sigma) : -double(sigma);
    return launch_streams(p, 1, &seed, &coef, static_cast<hipStream_t>(stream));
}

int check_qdevice(const es_qplan_t* p) {
    int dev = -1;
    const hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != p->device)
        return fail(ES_ERR_DEVICE, "current device " + std::to_string(dev) +
                                       " differs from the plan's device " +
                                       std::to_string(p->device));
    return ES_OK;
}

int launch_qpass(es_qplan_t* p, QKind kind, const QPass& ps, hipStream_t s) {
    if (p->n_full + p->n_tail == 0) return ES_OK;
    const QPassKernel kernel = qpass_kernel(p->threads, p->groups, kind, p->format);
    hipLaunchKernelGGL(kernel, dim3(p->grid), dim3(p->threads), 0, s, p->d_tab, p->n_full,
                       p->n_tail, reinterpret_cast<const Member*>(p->d_scratch + kOffMembers),
                       reinterpret_cast<const UpdateHeader*>(p->d_scratch + kOffHeader), ps);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "es_qpass_kernel launch");
    return ES_OK;
}

// The kernel argument of one perturbation member of a quantized pass: its
// key and sign * sigma * sqrt(2 ln 2) (a restore negates in the kernel).
Member qmember(uint64_t seed, int32_t sign, float sigma) {
    const double coef = sign > 0 ? double(sigma) : -double(sigma);
    return Member{static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32),
                  static_cast<float>(coef * kSqrt2Ln2Double), 0u};
}

int qperturb_impl(es_qplan_t* p, uint64_t seed, int32_t sign, float sigma, es_stream_t stream,
                  QKind kind, const char* name) {
    if (p == nullptr) return fail(ES_ERR_INVALID_ARG, std::string(name) + ": null plan");
    if (sign != 1 && sign != -1)
        return fail(ES_ERR_INVALID_ARG, std::string(name) + ": sign must be +1 or -1");
    if (!std::isfinite(sigma) || sigma < 0.0f)
        return fail(ES_ERR_INVALID_ARG, std::string(name) + ": sigma must be finite and >= 0");
    if (sigma == 0.0f) return ES_OK;
    const int rc = check_qdevice(p);
    if (rc != ES_OK) return rc;
    QPass ps = {};
    ps.m = qmember(seed, sign, sigma);
    return launch_qpass(p, kind, ps, static_cast<hipStream_t>(stream));
}

// The `bytes` bytes at p must be memory that kernels on `device` can access:
// device or managed memory of that device, the whole range inside one
// allocation (checked when the runtime knows the allocation's extent), or
// mapped pinned host memory.  Catches host pointers, other devices' memory
// and overstated sizes before a kernel would fault on them.  A failed query
// leaves no error behind for later launch checks.
// (The name of the checked array is `name` followed by `part`; it is
// formatted only on failure.)
int check_access(const void* p, uint64_t bytes, int device, const char* name, const char* part) {
    if (bytes == 0) return ES_OK;
    auto what = [&]() { return std::string(name) + part; };
    hipPointerAttribute_t a{};
    hipError_t e = hipPointerGetAttributes(&a, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(ES_ERR_INVALID_ARG, what() + ": not memory the device can access");
    }
    if (a.type == hipMemoryTypeHost) {
        if (a.devicePointer == nullptr)
            return fail(ES_ERR_INVALID_ARG, what() + ": host memory not mapped for the device");
        return ES_OK;
    }
    if (a.type != hipMemoryTypeDevice && a.type != hipMemoryTypeManaged &&
        a.type != hipMemoryTypeUnified)
        return fail(ES_ERR_INVALID_ARG, what() + ": not device memory");
    if (a.type == hipMemoryTypeDevice && a.device != device)
        return fail(ES_ERR_INVALID_ARG, what() + ": memory of device " + std::to_string(a.device) +
                                            ", not of device " + std::to_string(device));
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    e = hipMemGetAddressRange(&base, &size, const_cast<void*>(p));
    if (e != hipSuccess) {                   // allocator that does not report extents
        (void)hipGetLastError();
        return ES_OK;
    }
    const uintptr_t b = reinterpret_cast<uintptr_t>(base), q = reinterpret_cast<uintptr_t>(p);
    if (q < b || q - b > size || bytes > size - (q - b))
        return fail(ES_ERR_INVALID_ARG, what() + ": " + std::to_string(bytes) +
                                            " bytes extend past the end of its allocation");
    return ES_OK;
}
int check_access(const void* p, uint64_t bytes, int device, const std::string& what) {
    return check_access(p, bytes, device, what.c_str(), "");
}

// Free a plan's tile table and scratch on the plan's device: that device is made
// current for the call (the caller's is restored) and synchronised first, so
// no queued launch still reads them.  Every step runs; the first error is
// returned.
int release_device_memory(int device, void* tab, void* scratch, const char* name) {
    const std::string nm(name);
    int rc = ES_OK;
    int caller = -1;
    hipError_t e = hipGetDevice(&caller);
    if (e != hipSuccess) rc = hip_fail(e, nm + ": hipGetDevice");
    const bool switched = e == hipSuccess && caller != device;
    if (switched) {
        e = hipSetDevice(device);
        if (e != hipSuccess && rc == ES_OK) rc = hip_fail(e, nm + ": hipSetDevice");
    }
    e = hipDeviceSynchronize();
    if (e != hipSuccess && rc == ES_OK) rc = hip_fail(e, nm + ": hipDeviceSynchronize");
    e = hipFree(tab);
    if (e != hipSuccess && rc == ES_OK) rc = hip_fail(e, nm + ": hipFree");
    e = hipFree(scratch);
    if (e != hipSuccess && rc == ES_OK) rc = hip_fail(e, nm + ": hipFree");
    if (switched) {
        e = hipSetDevice(caller);
        if (e != hipSuccess && rc == ES_OK) rc = hip_fail(e, nm + ": hipSetDevice");
    }
    return rc;
}

// Division by a row length r >= 2 as a multiply-high and a shift:
// j / r = mulhi(j, magic) >> shift for every j < 2^31 (Granlund and
// Montgomery, 1994: magic = ceil(2^(31 + l) / r) with 2^(l-1) < r <= 2^l,
// which lies in [2^31, 2^32)).
void row_divisor(uint32_t r, uint32_t& magic, uint32_t& shift) {
    uint32_t l = 0;
    while ((uint64_t(1) << l) < r) ++l;
    magic = static_cast<uint32_t>(((uint64_t(1) << (31 + l)) + r - 1) / r);
    shift = l - 1;
}

// Launch shape of the bf16 tile kernels: the defaults, or overrides for
// launch-shape sweeps.
void launch_shape(int& threads, int& groups) {
    threads = env_int("ESOPT_THREADS", kDefaultThreads, 256, 1024);
    groups = env_int("ESOPT_GROUPS", kDefaultGroups, 2, 8);
    if (update_kernel(threads, groups, false, false) == nullptr) {
        threads = kDefaultThreads;
        groups = kDefaultGroups;
    }
}

// The tiles of one bf16 tensor (see DevTile), appended to `full` and `tail`.
// Full tiles start where the address is a multiple of the tile's byte size
// (the tensor's base is 16-byte aligned, so such an element index is a
// multiple of 8 and groups keep their Philox quads); the elements before the
// first one and after the last one are tail tiles.  A shard (`offset`
// elements into its whole tensor, a multiple of 8) is tiled by address the
// same way, but its descriptors count elements of the whole tensor: elem0
// and limit are offset, and the base is moved back by as many elements, so
// base + element is still the address and the element is the noise index.
// Every tile keeps its counter's high word uniform: a tile that would cross
// a multiple of 2^34 elements of the whole tensor is split there into tail
// tiles.
void tile_tensor(uint16_t* data, uint64_t numel, uint64_t offset, uint32_t tensor_id,
                 uint64_t tile_elems, std::vector<DevTile>& full, std::vector<DevTile>& tail) {
    if (numel == 0) return;
    constexpr uint64_t kHiBlock = uint64_t(1) << 34;      // elements per counter high word
    // base - offset, as an address: the kernels only ever add an element
    // index of at least `offset` to it
    uint16_t* const base =
        reinterpret_cast<uint16_t*>(reinterpret_cast<uintptr_t>(data) - 2 * offset);
    auto add_tail = [&](uint64_t e0, uint64_t e1, uint32_t aligned) {   // local indices
        e0 += offset;
        e1 += offset;
        while (e0 < e1) {                                   // split at high-word boundaries
            const uint64_t cut = std::min(e1, (e0 / kHiBlock + 1) * kHiBlock);
            tail.push_back(DevTile{base, e0, cut, tensor_id, aligned});
            e0 = cut;
        }
    };
    const uintptr_t a = reinterpret_cast<uintptr_t>(data);
    if (a % 16 != 0) {                                      // element-wise accesses throughout
        for (uint64_t e0 = 0; e0 < numel; e0 += tile_elems)
            add_tail(e0, std::min(numel, e0 + tile_elems), 0u);
        return;
    }
    const uint64_t tile_bytes = 2 * tile_elems;
    const uint64_t head = std::min<uint64_t>(numel, ((tile_bytes - a % tile_bytes) % tile_bytes) / 2);
    add_tail(0, head, 1u);
    uint64_t e0 = head;
    for (; e0 + tile_elems <= numel; e0 += tile_elems) {
        const uint64_t g0 = offset + e0;
        if (g0 / kHiBlock != (g0 + tile_elems - 1) / kHiBlock)
            add_tail(e0, e0 + tile_elems, 1u);
        else
            full.push_back(DevTile{base, g0, g0 + tile_elems, tensor_id, 1u});
    }
    add_tail(e0, numel, 1u);
}

int current_device(int* dev) {
    const hipError_t e = hipGetDevice(dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    return ES_OK;
}

// The device arrays of an update call: rewards and z (n floats), status.
int check_update_arrays(const char* name, int device, const float* rewards_dev, uint32_t n,
                        const float* z_out_dev, const int32_t* status_out_dev) {
    int rc = check_access(rewards_dev, uint64_t(4) * n, device, name, ": rewards");
    if (rc == ES_OK && z_out_dev != nullptr)
        rc = check_access(z_out_dev, uint64_t(4) * n, device, name, ": z output");
    if (rc == ES_OK && status_out_dev != nullptr)
        rc = check_access(status_out_dev, 4, device, name, ": status output");
    return rc;
}

// Argument checks shared by the update entry points.
int validate_update(const char* name, const uint64_t* seeds, const int32_t* signs,
                    const float* rewards_dev, uint32_t n_members, const es_update_opts_t* opts) {
    if (seeds == nullptr || signs == nullptr || rewards_dev == nullptr || opts == nullptr)
        return fail_in(ES_ERR_INVALID_ARG, name, "null pointer");
    if (n_members == 0 || n_members > ES_MAX_MEMBERS)
        return fail_in(ES_ERR_INVALID_ARG, name, "n_members out of range (1 .. 1024)");
    if ((opts->flags & ~(ES_UPDATE_DIV_SIGMA | ES_REWARDS_ARE_WEIGHTS |
                         ES_UPDATE_STOCHASTIC_ROUND | ES_UPDATE_MASTER)) != 0)
        return fail_in(ES_ERR_INVALID_ARG, name, "unknown flags");
    if ((opts->flags & ES_UPDATE_MASTER) && (opts->flags & ES_UPDATE_STOCHASTIC_ROUND))
        return fail_in(ES_ERR_INVALID_ARG, name,
                       "ES_UPDATE_MASTER rounds the bf16 copy to nearest-even: no "
                       "ES_UPDATE_STOCHASTIC_ROUND with it");
    if (!std::isfinite(opts->alpha)) return fail_in(ES_ERR_INVALID_ARG, name, "alpha not finite");
    if ((opts->flags & ES_UPDATE_DIV_SIGMA) && !(std::isfinite(opts->sigma) && opts->sigma > 0.0f))
        return fail_in(ES_ERR_INVALID_ARG, name,
                       "sigma must be finite and > 0 with ES_UPDATE_DIV_SIGMA");
    if (!std::isfinite(opts->zscore_eps) || opts->zscore_eps < 0.0f)
        return fail_in(ES_ERR_INVALID_ARG, name, "zscore_eps must be finite and >= 0");
    for (uint32_t i = 0; i < n_members; ++i)
        if (signs[i] != 1 && signs[i] != -1)
            return fail_in(ES_ERR_INVALID_ARG, name, "signs must be +1 or -1");
    return ES_OK;
}

// The population as tables (host side, fixed arrays, no allocation):
// distinct seeds in order of first appearance, each with its members grouped
// in member order (CSR).  Members are sorted by (seed, index) in place, each
// run of one seed is a distinct seed whose first appearance is its smallest
// index, and the runs are ordered by that index.
struct MemberTables {
    MemberIn min[ES_MAX_MEMBERS];
    DistinctIn din[ES_MAX_MEMBERS];
    uint32_t n_distinct;
};

void build_member_tables(const uint64_t* seeds, const int32_t* signs, uint32_t n,
                         MemberTables& t) {
    struct SeedIndex {
        uint64_t seed;
        uint32_t index;
    };
    struct Run {
        uint32_t first, start, count;       // smallest member index, position in `order`, size
    };
    SeedIndex order[ES_MAX_MEMBERS];
    Run runs[ES_MAX_MEMBERS];
    for (uint32_t i = 0; i < n; ++i) order[i] = SeedIndex{seeds[i], i};
    std::sort(order, order + n, [](const SeedIndex& a, const SeedIndex& b) {
        return a.seed != b.seed ? a.seed < b.seed : a.index < b.index;
    });
    uint32_t nd = 0;
    for (uint32_t i = 0; i < n;) {
        uint32_t j = i + 1;
        while (j < n && order[j].seed == order[i].seed) ++j;
        runs[nd++] = Run{order[i].index, i, j - i};
        i = j;
    }
    std::sort(runs, runs + nd, [](const Run& a, const Run& b) { return a.first < b.first; });
    uint32_t pos = 0;
    for (uint32_t d = 0; d < nd; ++d) {
        const uint64_t sd = order[runs[d].start].seed;
        t.din[d] = DistinctIn{static_cast<uint32_t>(sd), static_cast<uint32_t>(sd >> 32), pos,
                              runs[d].count};
        for (uint32_t k = 0; k < runs[d].count; ++k) {
            const uint32_t m = order[runs[d].start + k].index;
            t.min[pos++] = MemberIn{m, signs[m]};
        }
    }
    t.n_distinct = nd;
}

// Hand the population to the device: the member tables are staged into the
// scratch through kernel arguments, then one wave z-scores the rewards and
// merges the weights per distinct seed, leaving the weighted member table
// and its header in the scratch.  Allocates nothing.  With `find`, *found is
// set to the distinct-table entry of seed *find before anything is launched
// (or the call fails with INVALID_ARG when no member has that seed).
// Host words into device scratch at dst_off, in launches of es_stage_kernel
// carrying 1 KB of kernel arguments each (no staging buffer, no host
// synchronisation).
int stage_words(uint8_t* d_scratch, size_t dst_off, const void* src, size_t bytes,
                hipStream_t s) {
    const uint32_t* words = static_cast<const uint32_t*>(src);
    const size_t n_words = bytes / 4;
    for (size_t w0 = 0; w0 < n_words; w0 += kStageWords) {
        StageChunk chunk;
        const uint32_t nw = static_cast<uint32_t>(std::min<size_t>(kStageWords, n_words - w0));
        std::memcpy(chunk.words, words + w0, nw * 4);
        hipLaunchKernelGGL(es_stage_kernel, dim3(1), dim3(kAuxBlock), 0, s,
                           reinterpret_cast<uint32_t*>(d_scratch + dst_off) + w0, nw, chunk);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(e, "es_stage_kernel launch");
    }
    return ES_OK;
}

int prepare_update(uint8_t* d_scratch, const uint64_t* seeds, const int32_t* signs,
                   const float* rewards_dev, uint32_t n_members, const es_update_opts_t* opts,
                   float* z_out_dev, int32_t* status_out_dev, hipStream_t s,
                   const uint64_t* find = nullptr, uint32_t* found = nullptr) {
    MemberTables t;
    build_member_tables(seeds, signs, n_members, t);
    const uint32_t nd = t.n_distinct;
    if (find != nullptr) {
        uint32_t d = 0;
        while (d < nd && (uint64_t(t.din[d].k0) | (uint64_t(t.din[d].k1) << 32)) != *find) ++d;
        if (d == nd)
            return fail(ES_ERR_INVALID_ARG,
                        "es_restore_update: the restored member's seed is not among the seeds");
        *found = d;
    }

    auto stage = [&](size_t dst_off, const void* src, size_t bytes) -> int {
        return stage_words(d_scratch, dst_off, src, bytes, s);
    };
    int rc = stage(kOffMembersIn, t.min, sizeof(MemberIn) * n_members);
    if (rc == ES_OK) rc = stage(kOffDistinctIn, t.din, sizeof(DistinctIn) * nd);
    if (rc != ES_OK) return rc;

    double c = static_cast<double>(opts->alpha) / static_cast<double>(n_members);
    if (opts->flags & ES_UPDATE_DIV_SIGMA) c /= static_cast<double>(opts->sigma);
    hipLaunchKernelGGL(es_prepare_kernel, dim3(1), dim3(64), 0, s, rewards_dev, n_members,
                       static_cast<double>(opts->zscore_eps), opts->flags, c,
                       reinterpret_cast<const MemberIn*>(d_scratch + kOffMembersIn),
                       reinterpret_cast<const DistinctIn*>(d_scratch + kOffDistinctIn), nd,
                       reinterpret_cast<Member*>(d_scratch + kOffMembers),
                       reinterpret_cast<UpdateHeader*>(d_scratch + kOffHeader), z_out_dev,
                       status_out_dev);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "es_prepare_kernel launch");
    return ES_OK;
}

// The member es_restore_update reverts: its seed and the perturbation
// coefficient es_restore would apply (-sign sigma).
struct RestoreMember {
    uint64_t seed;
    double coef;
};

// The fused update of a bf16 plan with its member tables in `d_scratch`
// (the plan's, or the static array of es_update_noalloc); with `restore`,
// that member reverted in the same pass.
int update_impl(const char* name, es_plan_t* plan, uint8_t* d_scratch, const uint64_t* seeds,
                const int32_t* signs, const float* rewards_dev, uint32_t n_members,
                const es_update_opts_t* opts, float* z_out_dev, int32_t* status_out_dev,
                hipStream_t s, const RestoreMember* restore = nullptr) {
    if (opts->flags & ES_UPDATE_MASTER) {
        if (restore != nullptr)
            return fail_in(ES_ERR_INVALID_ARG, name,
                           "ES_UPDATE_MASTER rewrites the bf16 values from the masters, so no "
                           "member needs reverting first: use es_update");
        if (plan->d_master == nullptr)
            return fail_in(ES_ERR_INVALID_ARG, name,
                           "ES_UPDATE_MASTER on a plan without masters (es_plan_set_master)");
    }
    RestoreArg rst{0u, 0.0f};
    int rc = prepare_update(d_scratch, seeds, signs, rewards_dev, n_members, opts, z_out_dev,
                            status_out_dev, s, restore ? &restore->seed : nullptr, &rst.d);
    if (rc != ES_OK) return rc;
    if (restore) rst.coef_k = static_cast<float>(restore->coef * kSqrt2Ln2Double);
    const bool sr = (opts->flags & ES_UPDATE_STOCHASTIC_ROUND) != 0;
    const bool master = (opts->flags & ES_UPDATE_MASTER) != 0;
    const RoundKey rk{static_cast<uint32_t>(opts->round_seed),
                      static_cast<uint32_t>(opts->round_seed >> 32)};
    Segment seg[2];
    const int n_seg = plan_segments(plan, seg);
    for (int k = 0; k < n_seg; ++k) {
        const Segment& g = seg[k];
        const bool strided = g.rows != nullptr;
        const UpdateKernel kernel =
            master ? update_master_kernel(plan->threads, plan->groups, strided)
                   : update_kernel(plan->threads, plan->groups, sr, strided, restore != nullptr);
        // the segment's masters: the delta table runs parallel to the tiles
        const uint64_t* mdelta =
            master ? plan->d_master + (strided ? plan->n_full + plan->n_tail : 0) : nullptr;
        hipLaunchKernelGGL(kernel, dim3(g.grid_update), dim3(plan->threads), 0, s, g.tiles,
                           g.n_full, g.n_tail, g.rows,
                           reinterpret_cast<const Member*>(d_scratch + kOffMembers),
                           reinterpret_cast<const UpdateHeader*>(d_scratch + kOffHeader), rk,
                           rst, mdelta);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(e, std::string(name) + ": es_update_kernel launch");
    }
    return ES_OK;
}

// Per-device address of the static scratch, looked up once per device (with
// that device current) and kept; a fixed table, so lookups allocate nothing.
constexpr int kMaxScratchDevices = 64;
std::atomic<uint8_t*> g_static_scratch[kMaxScratchDevices];
std::mutex g_static_scratch_mutex;

int static_scratch(int device, uint8_t** out) {
    if (device < 0 || device >= kMaxScratchDevices)
        return fail_in(ES_ERR_DEVICE, "es_update_noalloc", "device index above 63");
    uint8_t* p = g_static_scratch[device].load(std::memory_order_acquire);
    if (p == nullptr) {
        std::lock_guard<std::mutex> lock(g_static_scratch_mutex);
        p = g_static_scratch[device].load(std::memory_order_relaxed);
        if (p == nullptr) {
            void* addr = nullptr;
            const hipError_t e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
            if (e != hipSuccess || addr == nullptr)
                return hip_fail(e, "es_update_noalloc: hipGetSymbolAddress of the static scratch");
            p = static_cast<uint8_t*>(addr);
            g_static_scratch[device].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return ES_OK;
}

// The tiles of a plan under construction: those of tensors and contiguous
// blocks, and those of strided blocks with one row map each.
struct PlanTiles {
    std::vector<DevTile> full, tail;
    std::vector<DevTile> rfull, rtail;
    std::vector<DevRows> rows_full, rows_tail;
};

// Strided blocks are cut into pieces of at most this many elements, so that
// a piece's local element indices stay below 2^31 (the row division's
// range).  A block whose rows are longer than half of that, or whose rows lie
// 2^32 or more elements apart, is laid out row by row instead, each row a
// contiguous shard of its own.
constexpr uint64_t kPieceElems = uint64_t(1) << 31;

// Appends a tile of a strided piece with its row map, cut into tail tiles
// where the whole-tensor index reaches a multiple of 2^34 (so that the
// counter's high word is the tile's).  Such a multiple lies at the start of
// a group: indices within a row are consecutive from a multiple of 8 and
// rows start at multiples of 8.  The index is increasing in e, so each cut
// is found by bisection over the tile's groups.
void split_at_high_words(const DevTile& d, DevRows m, bool full, PlanTiles& t) {
    constexpr uint64_t kHiBlock = uint64_t(1) << 34;
    auto index = [&](uint64_t e) { return rows_index(m.n0, m.skip, m.magic, m.shift, e); };
    uint64_t e0 = d.elem0;
    const uint64_t hi_last = index(d.limit - 1) / kHiBlock;
    if (index(e0) / kHiBlock == hi_last) {
        m.hi = static_cast<uint32_t>(hi_last);
        (full ? t.rfull : t.rtail).push_back(d);
        (full ? t.rows_full : t.rows_tail).push_back(m);
        return;
    }
    while (e0 < d.limit) {
        const uint64_t hi = index(e0) / kHiBlock;
        uint64_t lo_g = (e0 - d.elem0) / 8, hi_g = (d.limit - d.elem0 + 7) / 8;  // groups
        while (lo_g + 1 < hi_g) {          // last group of [e0, ...) still on `hi`
            const uint64_t mid = (lo_g + hi_g) / 2;
            if (index(d.elem0 + 8 * mid) / kHiBlock == hi) lo_g = mid;
            else hi_g = mid;
        }
        const uint64_t cut = std::min(d.limit, d.elem0 + 8 * hi_g);
        DevTile part = d;
        part.elem0 = e0;
        part.limit = cut;
        m.hi = static_cast<uint32_t>(hi);
        t.rtail.push_back(part);
        t.rows_tail.push_back(m);
        e0 = cut;
    }
}

// Tiles of one block (already validated).  A block that is one contiguous
// range of its tensor is tiled as a shard at its first index.  A strided
// block is cut into pieces of whole rows, each tiled by address with local
// element indices, and every tile of a piece gets the piece's row map.
void tile_block(const es_block_t& b, uint64_t tile_elems, PlanTiles& t) {
    const uint64_t numel = b.rows * b.cols;
    if (numel == 0) return;
    uint16_t* const data = static_cast<uint16_t*>(b.data);
    const uint64_t n0 = b.row0 * b.row_len + b.col0;
    if (b.rows == 1 || b.cols == b.row_len) {
        tile_tensor(data, numel, n0, b.tensor_id, tile_elems, t.full, t.tail);
        return;
    }
    if (b.cols > kPieceElems / 2 || b.row_len - b.cols > 0xFFFFFFFFull) {
        for (uint64_t i = 0; i < b.rows; ++i)
            tile_tensor(data + i * b.cols, b.cols, n0 + i * b.row_len, b.tensor_id, tile_elems,
                        t.full, t.tail);
        return;
    }
    DevRows m{};
    m.skip = static_cast<uint32_t>(b.row_len - b.cols);
    row_divisor(static_cast<uint32_t>(b.cols), m.magic, m.shift);
    const uint64_t piece_rows = kPieceElems / b.cols;
    std::vector<DevTile> full, tail;
    for (uint64_t r = 0; r < b.rows; r += piece_rows) {
        const uint64_t nr = std::min(piece_rows, b.rows - r);
        m.n0 = n0 + r * b.row_len;
        full.clear();
        tail.clear();
        tile_tensor(data + r * b.cols, nr * b.cols, 0, b.tensor_id, tile_elems, full, tail);
        for (int k = 0; k < 2; ++k)
            for (const DevTile& d : k == 0 ? full : tail) split_at_high_words(d, m, k == 0, t);
    }
}

// A plan over tiles laid out by the caller (es_plan_create,
// es_plan_create_blocks): launch grids, one device allocation for the
// descriptors and row maps, the scratch.
int finish_plan(const char* name, int device, uint32_t n_tensors, uint64_t numel, int threads,
                int groups, PlanTiles& t, es_plan_t** out) {
    const std::string nm(name);
    const uint64_t n_full = t.full.size(), n_tail = t.tail.size();
    const uint64_t n_rfull = t.rfull.size(), n_rtail = t.rtail.size();
    std::vector<DevTile> tiles;
    tiles.reserve(n_full + n_tail + n_rfull + n_rtail);
    tiles.insert(tiles.end(), t.full.begin(), t.full.end());
    tiles.insert(tiles.end(), t.tail.begin(), t.tail.end());
    tiles.insert(tiles.end(), t.rfull.begin(), t.rfull.end());
    tiles.insert(tiles.end(), t.rtail.begin(), t.rtail.end());
    std::vector<DevRows> rows;
    rows.reserve(n_rfull + n_rtail);
    rows.insert(rows.end(), t.rows_full.begin(), t.rows_full.end());
    rows.insert(rows.end(), t.rows_tail.begin(), t.rows_tail.end());
    es_plan_t* p = new (std::nothrow) es_plan_t;
    if (p == nullptr) return fail(ES_ERR_NOMEM, nm + ": host allocation");
    p->device = device;
    int cus = 0;
    hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, p->device);
    if (e != hipSuccess) { delete p; return hip_fail(e, "hipDeviceGetAttribute"); }
    const int wg_perturb = env_int("ESOPT_PERTURB_WG_PER_CU", kDefaultPerturbWgPerCu, 1, 32);
    const int wg_update = env_int("ESOPT_UPDATE_WG_PER_CU", kDefaultUpdateWgPerCu, 1, 32);
    p->threads = threads;
    p->groups = groups;
    p->tile_elems = uint64_t(threads) * groups * kGroupElems;
    p->n_tensors = n_tensors;
    p->numel = numel;
    p->n_full = n_full;
    p->n_tail = n_tail;
    p->n_rfull = n_rfull;
    p->n_rtail = n_rtail;
    auto grid = [&](uint64_t a, uint64_t b, int per_cu) {
        const uint64_t cap = std::max<uint64_t>(std::max(a, b), 1);
        return static_cast<uint32_t>(std::min<uint64_t>(cap, uint64_t(cus) * per_cu));
    };
    p->grid_perturb = grid(n_full, n_tail, wg_perturb);
    p->grid_update = grid(n_full, n_tail, wg_update);
    p->grid_perturb_rows = grid(n_rfull, n_rtail, wg_perturb);
    p->grid_update_rows = grid(n_rfull, n_rtail, wg_update);
    const size_t tile_bytes = sizeof(DevTile) * std::max<size_t>(tiles.size(), 1);
    const size_t rows_bytes = sizeof(DevRows) * rows.size();
    e = hipMalloc(reinterpret_cast<void**>(&p->d_tiles), tile_bytes + rows_bytes);
    if (e != hipSuccess) { delete p; return fail(ES_ERR_NOMEM, std::string("hipMalloc: ") + hipGetErrorString(e)); }
    p->d_rows = rows.empty() ? nullptr
                             : reinterpret_cast<DevRows*>(reinterpret_cast<uint8_t*>(p->d_tiles) +
                                                          tile_bytes);
    e = hipMalloc(reinterpret_cast<void**>(&p->d_scratch), kScratchBytes);
    if (e != hipSuccess) {
        (void)hipFree(p->d_tiles);
        delete p;
        return fail(ES_ERR_NOMEM, std::string("hipMalloc: ") + hipGetErrorString(e));
    }
    if (!tiles.empty())
        e = hipMemcpy(p->d_tiles, tiles.data(), sizeof(DevTile) * tiles.size(), hipMemcpyHostToDevice);
    if (e == hipSuccess && !rows.empty())
        e = hipMemcpy(p->d_rows, rows.data(), rows_bytes, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemset(p->d_scratch, 0, kScratchBytes);
    if (e != hipSuccess) {
        (void)hipFree(p->d_tiles);
        (void)hipFree(p->d_scratch);
        delete p;
        return hip_fail(e, nm + ": tile table upload");
    }
    *out = p;
    return ES_OK;
}

// Checks of one block's geometry (es_block_t's requirements), in 128-bit
// arithmetic so that no product or sum wraps; an empty string when it holds.
std::string block_geometry_error(const es_block_t& b) {
    typedef unsigned __int128 u128;
    const u128 two60 = u128(1) << 60;
    const u128 numel = u128(b.rows) * b.cols;
    if (numel > two60) return "rows * cols above 2^60";
    if (numel == 0) return "";
    if (u128(b.col0) + b.cols > b.row_len) return "col0 + cols above row_len";
    const u128 first = u128(b.row0) * b.row_len + b.col0;
    const u128 end = u128(b.row0 + u128(b.rows - 1)) * b.row_len + b.col0 + b.cols;
    if (end > two60) return "an element index at or above 2^60";
    if (first % 8 != 0) return "first index row0 * row_len + col0 not a multiple of 8";
    if (b.rows > 1 && b.cols < b.row_len && (b.cols % 8 != 0 || b.row_len % 8 != 0))
        return "strided block: cols and row_len must be multiples of 8";
    return "";
}


// One entry of a quantized plan, from an es_qtensor_t (with a shard start)
// or an es_qblock_t: `numel` codes at `data` with their scales, the
// whole-tensor index n0 of code 0 and, for a strided block, rows of `cols`
// codes that lie cols + skip apart in the whole tensor (skip 0 otherwise).
struct QSpec {
    void* data;
    const float* scales;
    uint64_t numel;
    uint32_t row, tensor_id;
    uint64_t n0, cols, skip;
};

// The geometry of a quantized block as a QSpec, or what is wrong with it.
std::string qblock_geometry(const es_qblock_t& b, QSpec& spec) {
    typedef unsigned __int128 u128;
    const u128 two31 = u128(1) << 31;
    const u128 numel = u128(b.rows) * b.cols;
    if (numel >= two31) return "rows * cols must be below 2^31";
    spec = QSpec{b.data, b.scales, uint64_t(numel), b.row, b.tensor_id, 0, b.cols, 0};
    if (numel == 0) return "";
    if (u128(b.col0) + b.cols > b.row_len) return "col0 + cols above row_len";
    const u128 first = u128(b.row0) * b.row_len + b.col0;
    const u128 end = (u128(b.row0) + b.rows - 1) * b.row_len + b.col0 + b.cols;
    if (end >= two31) return "(row0 + rows - 1) * row_len + col0 + cols must be below 2^31";
    if (first % 16 != 0) return "first index row0 * row_len + col0 not a multiple of 16";
    const bool strided = b.rows > 1 && b.cols < b.row_len;
    if (strided && (b.cols % 16 != 0 || b.row_len % 16 != 0))
        return "strided block: cols and row_len must be multiples of 16";
    spec.n0 = uint64_t(first);
    spec.skip = strided ? b.row_len - b.cols : 0;
    return "";
}

// A quantized plan over checked entries (whole-tensor indices below 2^31):
// the per-entry rules shared by tensors and blocks, the table, the device
// checks and the allocations.  `name` and `kind` label the errors.
int qplan_build(const std::vector<QSpec>& specs, uint32_t format, es_qplan_t** out,
                const char* name, const char* kind) {
    const std::string nm(name);
    if (format != ES_QFORMAT_INT8 && format != ES_QFORMAT_E4M3)
        return fail(ES_ERR_INVALID_ARG, nm + ": format not ES_QFORMAT_INT8 or ES_QFORMAT_E4M3");
    int threads = env_int("ESOPT_THREADS", kDefaultThreads, 256, 1024);
    int groups = env_int("ESOPT_QGROUPS", kDefaultQGroups, 2, 8);
    if (qpass_kernel(threads, groups, QKind::kUpdate, static_cast<int>(format)) == nullptr) {
        threads = kDefaultThreads;
        groups = kDefaultQGroups;
    }
    const uint64_t tile_elems = uint64_t(threads) * groups * esq::kQGroup;
    const uint32_t n_tensors = static_cast<uint32_t>(specs.size());
    std::vector<esq::DevQTensor> tab(n_tensors + 1);
    std::unordered_map<uint32_t, uint32_t> ids;
    std::vector<std::pair<uintptr_t, uintptr_t>> ranges;
    uint64_t n_full = 0, n_tail = 0, numel = 0;
    for (uint32_t i = 0; i < n_tensors; ++i) {
        const QSpec& t = specs[i];
        const std::string where = nm + ": " + kind + " " + std::to_string(i);
        if (!ids.emplace(t.tensor_id, i).second)
            return fail(ES_ERR_INVALID_ARG, where + ": duplicate tensor_id " + std::to_string(t.tensor_id));
        if (t.numel > 0 && (t.data == nullptr || t.scales == nullptr))
            return fail(ES_ERR_INVALID_ARG, where + ": null data or scales");
        if (t.row % 8 != 0)
            return fail(ES_ERR_INVALID_ARG, where + ": row must be a multiple of 8 (or 0)");
        if (t.numel > 0 && (reinterpret_cast<uintptr_t>(t.scales) & 3u))
            return fail(ES_ERR_ALIGN, where + ": scales not 4-byte aligned");
        const uintptr_t a = reinterpret_cast<uintptr_t>(t.data);
        const uint64_t full = (a % 16 == 0) ? t.numel / tile_elems : 0;
        const uint64_t tail = (t.numel - full * tile_elems + tile_elems - 1) / tile_elems;
        uint32_t magic = 0, shift = 0, cmagic = 0, cshift = 0;
        if (t.row != 0) row_divisor(t.row, magic, shift);
        if (t.skip != 0) row_divisor(static_cast<uint32_t>(t.cols), cmagic, cshift);
        tab[i] = esq::DevQTensor{static_cast<int8_t*>(t.data), t.scales,
                                 static_cast<uint32_t>(t.numel), static_cast<uint32_t>(t.n0),
                                 n_full, n_tail, t.row, t.tensor_id, magic, shift, n_tensors,
                                 (a % 16 == 0) ? 1u : 0u, static_cast<uint32_t>(t.skip), cmagic,
                                 cshift, 0u};
        if (t.numel > 0) ranges.emplace_back(a, a + t.numel);
        n_full += full;
        n_tail += tail;
        numel += t.numel;
    }
    std::sort(ranges.begin(), ranges.end());
    for (size_t i = 1; i < ranges.size(); ++i)
        if (ranges[i].first < ranges[i - 1].second)
            return fail(ES_ERR_INVALID_ARG, nm + ": " + kind + "s overlap in memory");
    tab[n_tensors] = esq::DevQTensor{nullptr, nullptr, 0u, 0u, n_full, n_tail, 0u, 0xFFFFFFFFu,
                                     0u, 0u, n_tensors, 0u, 0u, 0u, 0u, 0u};

    int device = -1;
    int rc = current_device(&device);
    if (rc != ES_OK) return rc;
    for (uint32_t i = 0; i < n_tensors && rc == ES_OK; ++i) {
        const QSpec& t = specs[i];
        const std::string where = nm + ": " + kind + " " + std::to_string(i);
        const uint64_t n_scales = t.row == 0 ? 1 : (t.numel + t.row - 1) / t.row;
        rc = check_access(t.data, t.numel, device, where + " codes");
        if (rc == ES_OK && t.numel > 0)
            rc = check_access(t.scales, 4 * n_scales, device, where + " scales");
    }
    if (rc != ES_OK) return rc;
    es_qplan_t* p = new (std::nothrow) es_qplan_t;
    if (p == nullptr) return fail(ES_ERR_NOMEM, nm + ": host allocation");
    p->device = device;
    hipError_t e = hipSuccess;
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, p->device);
    if (e != hipSuccess) { delete p; return hip_fail(e, "hipDeviceGetAttribute"); }
    const int wg = env_int("ESOPT_UPDATE_WG_PER_CU", kDefaultUpdateWgPerCu, 1, 32);
    p->threads = threads;
    p->groups = groups;
    p->format = static_cast<int>(format);
    p->n_tensors = n_tensors;
    p->numel = numel;
    p->n_full = n_full;
    p->n_tail = n_tail;
    const uint64_t cap = std::max<uint64_t>(std::max(n_full, n_tail), 1);
    p->grid = static_cast<uint32_t>(std::min<uint64_t>(cap, uint64_t(cus) * wg));
    e = hipMalloc(reinterpret_cast<void**>(&p->d_tab), sizeof(esq::DevQTensor) * tab.size());
    if (e != hipSuccess) { delete p; return fail(ES_ERR_NOMEM, std::string("hipMalloc: ") + hipGetErrorString(e)); }
    e = hipMalloc(reinterpret_cast<void**>(&p->d_scratch), kScratchBytes);
    if (e != hipSuccess) {
        (void)hipFree(p->d_tab);
        delete p;
        return fail(ES_ERR_NOMEM, std::string("hipMalloc: ") + hipGetErrorString(e));
    }
    e = hipMemcpy(p->d_tab, tab.data(), sizeof(esq::DevQTensor) * tab.size(), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemset(p->d_scratch, 0, kScratchBytes);
    if (e != hipSuccess) {
        (void)hipFree(p->d_tab);
        (void)hipFree(p->d_scratch);
        delete p;
        return hip_fail(e, nm + ": table upload");
    }
    *out = p;
    return ES_OK;
}

}  // namespace

extern "C" {

int es_plan_create(const es_tensor_t* tensors, uint32_t n_tensors, es_plan_t** out) try {
    if (out == nullptr) return fail(ES_ERR_INVALID_ARG, "es_plan_create: null output pointer");
    *out = nullptr;
    if (tensors == nullptr) return fail(ES_ERR_INVALID_ARG, "es_plan_create: null tensor list");
    if (n_tensors == 0 || n_tensors > ES_MAX_TENSORS)
        return fail(ES_ERR_INVALID_ARG, "es_plan_create: n_tensors out of range");
    int threads = 0, groups = 0;
    launch_shape(threads, groups);
    const uint64_t tile_elems = uint64_t(threads) * groups * kGroupElems;
    std::unordered_map<uint32_t, uint32_t> ids;
    std::vector<std::pair<uintptr_t, uintptr_t>> ranges;
    uint64_t numel = 0;
    for (uint32_t i = 0; i < n_tensors; ++i) {
        const es_tensor_t& t = tensors[i];
        const std::string where = "es_plan_create: tensor " + std::to_string(i);
        if (!ids.emplace(t.tensor_id, i).second)
            return fail(ES_ERR_INVALID_ARG, where + ": duplicate tensor_id " + std::to_string(t.tensor_id));
        if (t.numel > 0 && t.data == nullptr) return fail(ES_ERR_INVALID_ARG, where + ": null data");
        if (t.numel > (uint64_t(1) << 60) - 8 * uint64_t(t.offset8))
            return fail(ES_ERR_INVALID_ARG, where + ": 8 * offset8 + numel above 2^60");
        const uintptr_t a = reinterpret_cast<uintptr_t>(t.data);
        if (t.numel > 0 && (a & 1u)) return fail(ES_ERR_ALIGN, where + ": data not 2-byte aligned");
        if (t.numel > 0) ranges.emplace_back(a, a + 2 * t.numel);
        numel += t.numel;
    }
    std::sort(ranges.begin(), ranges.end());
    for (size_t i = 1; i < ranges.size(); ++i)
        if (ranges[i].first < ranges[i - 1].second)
            return fail(ES_ERR_INVALID_ARG, "es_plan_create: tensors overlap in memory");

    int device = -1;
    int rc = current_device(&device);
    if (rc != ES_OK) return rc;
    for (uint32_t i = 0; i < n_tensors && rc == ES_OK; ++i)
        rc = check_access(tensors[i].data, 2 * tensors[i].numel, device,
                          "es_plan_create: tensor " + std::to_string(i));
    if (rc != ES_OK) return rc;
    // the tile descriptors (built after the accesses are known to be valid:
    // every tensor lies inside one device allocation)
    PlanTiles t;
    for (uint32_t i = 0; i < n_tensors; ++i)
        tile_tensor(static_cast<uint16_t*>(tensors[i].data), tensors[i].numel,
                    8 * uint64_t(tensors[i].offset8), tensors[i].tensor_id, tile_elems, t.full,
                    t.tail);
    rc = finish_plan("es_plan_create", device, n_tensors, numel, threads, groups, t, out);
    if (rc == ES_OK)
        for (uint32_t i = 0; i < n_tensors; ++i)
            (*out)->owners.emplace_back(reinterpret_cast<uintptr_t>(tensors[i].data),
                                        tensors[i].numel);
    return rc;
} catch (const std::bad_alloc&) {
    return fail(ES_ERR_NOMEM, "es_plan_create: host allocation failed");
}

int es_plan_create_blocks(const es_block_t* blocks, uint32_t n_blocks, es_plan_t** out) try {
    if (out == nullptr) return fail(ES_ERR_INVALID_ARG, "es_plan_create_blocks: null output pointer");
    *out = nullptr;
    if (blocks == nullptr) return fail(ES_ERR_INVALID_ARG, "es_plan_create_blocks: null block list");
    if (n_blocks == 0 || n_blocks > ES_MAX_TENSORS)
        return fail(ES_ERR_INVALID_ARG, "es_plan_create_blocks: n_blocks out of range");
    int threads = 0, groups = 0;
    launch_shape(threads, groups);
    const uint64_t tile_elems = uint64_t(threads) * groups * kGroupElems;
    std::unordered_map<uint32_t, uint32_t> ids;
    std::vector<std::pair<uintptr_t, uintptr_t>> ranges;
    uint64_t numel = 0;
    for (uint32_t i = 0; i < n_blocks; ++i) {
        const es_block_t& b = blocks[i];
        const std::string where = "es_plan_create_blocks: block " + std::to_string(i);
        if (b.reserved != 0) return fail(ES_ERR_INVALID_ARG, where + ": reserved field not 0");
        if (!ids.emplace(b.tensor_id, i).second)
            return fail(ES_ERR_INVALID_ARG, where + ": duplicate tensor_id " + std::to_string(b.tensor_id));
        const std::string bad = block_geometry_error(b);
        if (!bad.empty()) return fail(ES_ERR_INVALID_ARG, where + ": " + bad);
        const uint64_t n = b.rows * b.cols;
        if (n > 0 && b.data == nullptr) return fail(ES_ERR_INVALID_ARG, where + ": null data");
        const uintptr_t a = reinterpret_cast<uintptr_t>(b.data);
        if (n > 0 && (a & 1u)) return fail(ES_ERR_ALIGN, where + ": data not 2-byte aligned");
        if (n > 0) ranges.emplace_back(a, a + 2 * n);
        numel += n;
    }
    std::sort(ranges.begin(), ranges.end());
    for (size_t i = 1; i < ranges.size(); ++i)
        if (ranges[i].first < ranges[i - 1].second)
            return fail(ES_ERR_INVALID_ARG, "es_plan_create_blocks: blocks overlap in memory");

    int device = -1;
    int rc = current_device(&device);
    if (rc != ES_OK) return rc;
    for (uint32_t i = 0; i < n_blocks && rc == ES_OK; ++i)
        rc = check_access(blocks[i].data, 2 * blocks[i].rows * blocks[i].cols, device,
                          "es_plan_create_blocks: block " + std::to_string(i));
    if (rc != ES_OK) return rc;
    PlanTiles t;
    for (uint32_t i = 0; i < n_blocks; ++i) tile_block(blocks[i], tile_elems, t);
    rc = finish_plan("es_plan_create_blocks", device, n_blocks, numel, threads, groups, t, out);
    if (rc == ES_OK)
        for (uint32_t i = 0; i < n_blocks; ++i)
            (*out)->owners.emplace_back(reinterpret_cast<uintptr_t>(blocks[i].data),
                                        blocks[i].rows * blocks[i].cols);
    return rc;
} catch (const std::bad_alloc&) {
    return fail(ES_ERR_NOMEM, "es_plan_create_blocks: host allocation failed");
}

int es_plan_destroy(es_plan_t* plan) {
    if (plan == nullptr) return ES_OK;
    int rc = release_device_memory(plan->device, plan->d_tiles, plan->d_scratch,
                                   "es_plan_destroy");
    if (plan->d_master != nullptr) {
        const int rc2 = release_device_memory(plan->device, plan->d_master, nullptr,
                                              "es_plan_destroy");
        if (rc == ES_OK) rc = rc2;
    }
    delete plan;
    return rc;
}

int es_plan_set_master(es_plan_t* plan, void* const* masters, uint32_t n) try {
    if (plan == nullptr) return fail(ES_ERR_INVALID_ARG, "es_plan_set_master: null plan");
    if (masters == nullptr) {                         // detach
        if (plan->d_master == nullptr) return ES_OK;
        uint64_t* old = plan->d_master;
        plan->d_master = nullptr;
        return release_device_memory(plan->device, old, nullptr, "es_plan_set_master");
    }
    if (n != plan->owners.size())
        return fail(ES_ERR_INVALID_ARG, "es_plan_set_master: " + std::to_string(n) +
                                            " masters for a plan of " +
                                            std::to_string(plan->owners.size()) + " tensors");
    int rc = check_device(plan);
    if (rc != ES_OK) return rc;
    // validation: 16-byte aligned, inside one allocation of this device, and
    // overlapping no other master and no bf16 tensor of the plan
    std::vector<std::pair<uintptr_t, uintptr_t>> ranges;
    for (uint32_t i = 0; i < n; ++i) {
        const uint64_t numel = plan->owners[i].second;
        if (numel == 0) continue;
        const std::string where = "es_plan_set_master: master " + std::to_string(i);
        const uintptr_t a = reinterpret_cast<uintptr_t>(masters[i]);
        if (a == 0) return fail(ES_ERR_INVALID_ARG, where + ": null");
        if (a % 16 != 0) return fail(ES_ERR_ALIGN, where + ": not 16-byte aligned");
        rc = check_access(masters[i], 4 * numel, plan->device, where);
        if (rc != ES_OK) return rc;
        ranges.emplace_back(a, a + 4 * numel);
        ranges.emplace_back(plan->owners[i].first, plan->owners[i].first + 2 * numel);
    }
    std::sort(ranges.begin(), ranges.end());
    for (size_t i = 1; i < ranges.size(); ++i)
        if (ranges[i].first < ranges[i - 1].second)
            return fail(ES_ERR_INVALID_ARG,
                        "es_plan_set_master: masters overlap each other or the bf16 tensors");
    // each tile's owner: the tensor whose bf16 bytes hold the tile's first
    // element (tensors do not overlap), found by bisection over their starts
    const uint64_t n_tiles = plan->n_full + plan->n_tail + plan->n_rfull + plan->n_rtail;
    std::vector<DevTile> tiles(n_tiles);
    hipError_t e = hipSuccess;
    if (n_tiles > 0)
        e = hipMemcpy(tiles.data(), plan->d_tiles, sizeof(DevTile) * n_tiles,
                      hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "es_plan_set_master: tile table read-back");
    std::vector<std::pair<uintptr_t, uint32_t>> starts;      // (bf16 start, owner)
    for (uint32_t i = 0; i < n; ++i)
        if (plan->owners[i].second > 0) starts.emplace_back(plan->owners[i].first, i);
    std::sort(starts.begin(), starts.end());
    std::vector<uint64_t> delta(std::max<uint64_t>(n_tiles, 1), 0);
    for (uint64_t k = 0; k < n_tiles; ++k) {
        const uintptr_t first = reinterpret_cast<uintptr_t>(tiles[k].data) + 2 * tiles[k].elem0;
        auto it = std::upper_bound(starts.begin(), starts.end(),
                                   std::make_pair(first, std::numeric_limits<uint32_t>::max()));
        const uint32_t i = std::prev(it)->second;
        delta[k] = reinterpret_cast<uintptr_t>(masters[i]) - 2 * plan->owners[i].first;
    }
    uint64_t* d = nullptr;
    e = hipMalloc(reinterpret_cast<void**>(&d), sizeof(uint64_t) * delta.size());
    if (e != hipSuccess) return fail(ES_ERR_NOMEM, std::string("hipMalloc: ") + hipGetErrorString(e));
    e = hipMemcpy(d, delta.data(), sizeof(uint64_t) * delta.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(d);
        return hip_fail(e, "es_plan_set_master: table upload");
    }
    uint64_t* old = plan->d_master;
    plan->d_master = d;
    if (old != nullptr) return release_device_memory(plan->device, old, nullptr,
                                                     "es_plan_set_master");
    return ES_OK;
} catch (const std::bad_alloc&) {
    return fail(ES_ERR_NOMEM, "es_plan_set_master: host allocation failed");
}

int es_perturb_master(es_plan_t* plan, uint64_t seed, int32_t sign, float sigma,
                      es_stream_t stream) {
    if (plan == nullptr) return fail(ES_ERR_INVALID_ARG, "es_perturb_master: null plan");
    if (sign != 1 && sign != -1)
        return fail(ES_ERR_INVALID_ARG, "es_perturb_master: sign must be +1 or -1");
    if (!std::isfinite(sigma) || sigma < 0.0f)
        return fail(ES_ERR_INVALID_ARG, "es_perturb_master: sigma must be finite and >= 0");
    if (plan->d_master == nullptr)
        return fail(ES_ERR_INVALID_ARG, "es_perturb_master: the plan has no masters "
                                        "(es_plan_set_master)");
    int rc = check_device(plan);
    if (rc != ES_OK) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const double coef = sign > 0 ? double(sigma) : -double(sigma);
    Segment seg[2];
    const int n_seg = plan_segments(plan, seg);
    if (sigma != 0.0f) {
        Streams st = {};
        st.k0[0] = static_cast<uint32_t>(seed);
        st.k1[0] = static_cast<uint32_t>(seed >> 32);
        st.coef_k[0] = static_cast<float>(coef * kSqrt2Ln2Double);
        for (int k = 0; k < n_seg; ++k) {
            const Segment& g = seg[k];
            const bool strided = g.rows != nullptr;
            hipLaunchKernelGGL(apply_master_kernel(plan->threads, plan->groups, strided),
                               dim3(g.grid_perturb), dim3(plan->threads), 0, s, g.tiles, g.n_full,
                               g.n_tail, g.rows, st,
                               plan->d_master + (strided ? plan->n_full + plan->n_tail : 0));
            const hipError_t e = hipGetLastError();
            if (e != hipSuccess)
                return hip_fail(e, "es_perturb_master: es_apply_master_kernel launch");
        }
        return ES_OK;
    }
    // sigma == 0 rewrites the bf16 values as the masters rounded to nearest
    // even (-0 stays -0: no term is added): the update kernel's application
    // of members with a one-member table of zero weight in the plan's scratch
    const Member m{static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32),
                   static_cast<float>(coef * kSqrt2Ln2Double), 0u};
    const UpdateHeader h{1u, 0u, 0, 0u};
    rc = stage_words(plan->d_scratch, kOffMembers, &m, sizeof(m), s);
    if (rc == ES_OK) rc = stage_words(plan->d_scratch, kOffHeader, &h, sizeof(h), s);
    if (rc != ES_OK) return rc;
    for (int k = 0; k < n_seg; ++k) {
        const Segment& g = seg[k];
        const bool strided = g.rows != nullptr;
        hipLaunchKernelGGL(update_master_kernel(plan->threads, plan->groups, strided, true),
                           dim3(g.grid_update), dim3(plan->threads), 0, s, g.tiles, g.n_full,
                           g.n_tail, g.rows,
                           reinterpret_cast<const Member*>(plan->d_scratch + kOffMembers),
                           reinterpret_cast<const UpdateHeader*>(plan->d_scratch + kOffHeader),
                           RoundKey{0u, 0u}, RestoreArg{0u, 0.0f},
                           plan->d_master + (strided ? plan->n_full + plan->n_tail : 0));
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(e, "es_perturb_master: es_update_kernel launch");
    }
    return ES_OK;
}

uint64_t es_plan_numel(const es_plan_t* plan) { return plan ? plan->numel : 0; }

uint64_t es_plan_device_bytes(const es_plan_t* plan) {
    if (plan == nullptr) return 0;
    const uint64_t tiles =
        std::max<uint64_t>(plan->n_full + plan->n_tail + plan->n_rfull + plan->n_rtail, 1);
    return sizeof(DevTile) * tiles + sizeof(DevRows) * (plan->n_rfull + plan->n_rtail) +
           kScratchBytes + (plan->d_master != nullptr ? sizeof(uint64_t) * tiles : 0);
}
uint64_t es_plan_tiles(const es_plan_t* plan) {
    return plan ? plan->n_full + plan->n_tail + plan->n_rfull + plan->n_rtail : 0;
}

int es_perturb(es_plan_t* plan, uint64_t seed, int32_t sign, float sigma, es_stream_t stream) {
    return perturb_impl(plan, seed, sign, sigma, stream, "es_perturb");
}

int es_restore(es_plan_t* plan, uint64_t seed, int32_t sign, float sigma, es_stream_t stream) {
    if (sign != 1 && sign != -1)
        return fail(ES_ERR_INVALID_ARG, "es_restore: sign must be +1 or -1");
    return perturb_impl(plan, seed, -sign, sigma, stream, "es_restore");
}

int es_zscore(const float* rewards_dev, uint32_t n, float eps, float* z_dev, int32_t* status_dev,
              es_stream_t stream) {
    if (rewards_dev == nullptr || z_dev == nullptr)
        return fail(ES_ERR_INVALID_ARG, "es_zscore: null pointer");
    if (n == 0 || n > ES_MAX_MEMBERS) return fail(ES_ERR_INVALID_ARG, "es_zscore: n out of range");
    if (!std::isfinite(eps) || eps < 0.0f)
        return fail(ES_ERR_INVALID_ARG, "es_zscore: eps must be finite and >= 0");
    int device = -1;
    int rc = current_device(&device);
    if (rc == ES_OK) rc = check_update_arrays("es_zscore", device, rewards_dev, n, z_dev, status_dev);
    if (rc != ES_OK) return rc;
    hipLaunchKernelGGL(es_zscore_kernel, dim3(1), dim3(64), 0, static_cast<hipStream_t>(stream),
                       rewards_dev, n, static_cast<double>(eps), z_dev, status_dev);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "es_zscore_kernel launch");
    return ES_OK;
}

int es_update(es_plan_t* plan, const uint64_t* seeds, const int32_t* signs,
              const float* rewards_dev, uint32_t n_members, const es_update_opts_t* opts,
              float* z_out_dev, int32_t* status_out_dev, es_stream_t stream) try {
    if (plan == nullptr) return fail(ES_ERR_INVALID_ARG, "es_update: null plan");
    int rc = validate_update("es_update", seeds, signs, rewards_dev, n_members, opts);
    if (rc != ES_OK) return rc;
    rc = check_device(plan);
    if (rc == ES_OK)
        rc = check_update_arrays("es_update", plan->device, rewards_dev, n_members, z_out_dev,
                                 status_out_dev);
    if (rc != ES_OK) return rc;
    return update_impl("es_update", plan, plan->d_scratch, seeds, signs, rewards_dev, n_members,
                       opts, z_out_dev, status_out_dev, static_cast<hipStream_t>(stream));
} catch (const std::bad_alloc&) {
    return fail(ES_ERR_NOMEM, "es_update: host allocation failed");
}

int es_restore_update(es_plan_t* plan, uint64_t restore_seed, int32_t restore_sign,
                      float restore_sigma, const uint64_t* seeds, const int32_t* signs,
                      const float* rewards_dev, uint32_t n_members, const es_update_opts_t* opts,
                      float* z_out_dev, int32_t* status_out_dev, es_stream_t stream) try {
    if (plan == nullptr) return fail(ES_ERR_INVALID_ARG, "es_restore_update: null plan");
    if (restore_sign != 1 && restore_sign != -1)
        return fail(ES_ERR_INVALID_ARG, "es_restore_update: restore_sign must be +1 or -1");
    if (!std::isfinite(restore_sigma) || restore_sigma < 0.0f)
        return fail(ES_ERR_INVALID_ARG,
                    "es_restore_update: restore_sigma must be finite and >= 0");
    int rc = validate_update("es_restore_update", seeds, signs, rewards_dev, n_members, opts);
    if (rc != ES_OK) return rc;
    rc = check_device(plan);
    if (rc == ES_OK)
        rc = check_update_arrays("es_restore_update", plan->device, rewards_dev, n_members,
                                 z_out_dev, status_out_dev);
    if (rc != ES_OK) return rc;
    // es_restore with sigma 0 changes nothing: the update alone, as es_update
    const RestoreMember rm{restore_seed, restore_sign > 0 ? -double(restore_sigma)
                                                          : double(restore_sigma)};
    return update_impl("es_restore_update", plan, plan->d_scratch, seeds, signs, rewards_dev,
                       n_members, opts, z_out_dev, status_out_dev,
                       static_cast<hipStream_t>(stream), restore_sigma != 0.0f ? &rm : nullptr);
} catch (const std::bad_alloc&) {
    return fail(ES_ERR_NOMEM, "es_restore_update: host allocation failed");
}

int es_update_noalloc(es_plan_t* plan, const uint64_t* seeds, const int32_t* signs,
                      const float* rewards_dev, uint32_t n_members, const es_update_opts_t* opts,
                      float* z_out_dev, int32_t* status_out_dev, es_stream_t stream) try {
    if (plan == nullptr) return fail_in(ES_ERR_INVALID_ARG, "es_update_noalloc", "null plan");
    int rc = validate_update("es_update_noalloc", seeds, signs, rewards_dev, n_members, opts);
    if (rc != ES_OK) return rc;
    rc = check_device(plan);
    if (rc == ES_OK)
        rc = check_update_arrays("es_update_noalloc", plan->device, rewards_dev, n_members,
                                 z_out_dev, status_out_dev);
    uint8_t* d_scratch = nullptr;
    if (rc == ES_OK) rc = static_scratch(plan->device, &d_scratch);
    if (rc != ES_OK) return rc;
    return update_impl("es_update_noalloc", plan, d_scratch, seeds, signs, rewards_dev,
                       n_members, opts, z_out_dev, status_out_dev,
                       static_cast<hipStream_t>(stream));
} catch (const std::bad_alloc&) {
    return fail(ES_ERR_NOMEM, "es_update_noalloc: host allocation failed (error reporting)");
}

int es_swap(es_plan_t* plan, uint64_t seed_from, int32_t sign_from, float sigma_from,
            uint64_t seed_to, int32_t sign_to, float sigma_to, es_stream_t stream) {
    if (plan == nullptr) return fail(ES_ERR_INVALID_ARG, "es_swap: null plan");
    if ((sign_from != 1 && sign_from != -1) || (sign_to != 1 && sign_to != -1))
        return fail(ES_ERR_INVALID_ARG, "es_swap: signs must be +1 or -1");
    if (!std::isfinite(sigma_from) || sigma_from < 0.0f || !std::isfinite(sigma_to) ||
        sigma_to < 0.0f)
        return fail(ES_ERR_INVALID_ARG, "es_swap: sigmas must be finite and >= 0");
    // es_restore(from) then es_perturb(to); a zero sigma makes its half the
    // identity, as in those calls, and its stream is dropped.
    uint64_t sd[2];
    double cf[2];
    int m = 0;
    if (sigma_from != 0.0f) {
        sd[m] = seed_from;
        cf[m] = sign_from > 0 ? -double(sigma_from) : double(sigma_from);
        ++m;
    }
    if (sigma_to != 0.0f) {
        sd[m] = seed_to;
        cf[m] = sign_to > 0 ? double(sigma_to) : -double(sigma_to);
        ++m;
    }
    if (m == 0) return ES_OK;
    const int rc = check_device(plan);
    if (rc != ES_OK) return rc;
    const int streams = (m == 2 && sd[0] == sd[1]) ? 3 : m;
    return launch_streams(plan, streams, sd, cf, static_cast<hipStream_t>(stream));
}

int es_qplan_create(const es_qtensor_t* tensors, uint32_t n_tensors, es_qplan_t** out) {
    return es_qplan_create_format(tensors, n_tensors, ES_QFORMAT_INT8, out);
}

int es_qplan_create_format(const es_qtensor_t* tensors, uint32_t n_tensors, uint32_t format,
                           es_qplan_t** out) {
    return es_qplan_create_shards(tensors, nullptr, n_tensors, format, out);
}

int es_qplan_create_shards(const es_qtensor_t* tensors, const uint64_t* elem0, uint32_t n_tensors,
                           uint32_t format, es_qplan_t** out) try {
    if (out == nullptr) return fail(ES_ERR_INVALID_ARG, "es_qplan_create: null output pointer");
    *out = nullptr;
    if (tensors == nullptr) return fail(ES_ERR_INVALID_ARG, "es_qplan_create: null tensor list");
    if (n_tensors == 0 || n_tensors > ES_MAX_TENSORS)
        return fail(ES_ERR_INVALID_ARG, "es_qplan_create: n_tensors out of range");
    std::vector<QSpec> specs(n_tensors);
    for (uint32_t i = 0; i < n_tensors; ++i) {
        const es_qtensor_t& t = tensors[i];
        const std::string where = "es_qplan_create: tensor " + std::to_string(i);
        const uint64_t n0 = elem0 == nullptr ? 0 : elem0[i];
        if (t.numel >= (uint64_t(1) << 31))
            return fail(ES_ERR_INVALID_ARG, where + ": numel must be below 2^31");
        if (n0 >= (uint64_t(1) << 31) - t.numel)
            return fail(ES_ERR_INVALID_ARG, where + ": elem0 + numel must be below 2^31");
        if (n0 % 16 != 0)
            return fail(ES_ERR_INVALID_ARG, where + ": elem0 must be a multiple of 16");
        if (t.row != 0 && n0 % t.row != 0)
            return fail(ES_ERR_INVALID_ARG, where + ": elem0 must be a multiple of row");
        specs[i] = QSpec{t.data, t.scales, t.numel, t.row, t.tensor_id, n0, t.numel, 0};
    }
    return qplan_build(specs, format, out, "es_qplan_create", "tensor");
} catch (const std::bad_alloc&) {
    return fail(ES_ERR_NOMEM, "es_qplan_create: host allocation failed");
}

int es_qplan_create_blocks(const es_qblock_t* blocks, uint32_t n_blocks, uint32_t format,
                           es_qplan_t** out) try {
    if (out == nullptr) return fail(ES_ERR_INVALID_ARG, "es_qplan_create_blocks: null output pointer");
    *out = nullptr;
    if (blocks == nullptr) return fail(ES_ERR_INVALID_ARG, "es_qplan_create_blocks: null block list");
    if (n_blocks == 0 || n_blocks > ES_MAX_TENSORS)
        return fail(ES_ERR_INVALID_ARG, "es_qplan_create_blocks: n_blocks out of range");
    std::vector<QSpec> specs(n_blocks);
    for (uint32_t i = 0; i < n_blocks; ++i) {
        const std::string bad = qblock_geometry(blocks[i], specs[i]);
        if (!bad.empty())
            return fail(ES_ERR_INVALID_ARG,
                        "es_qplan_create_blocks: block " + std::to_string(i) + ": " + bad);
    }
    return qplan_build(specs, format, out, "es_qplan_create_blocks", "block");
} catch (const std::bad_alloc&) {
    return fail(ES_ERR_NOMEM, "es_qplan_create_blocks: host allocation failed");
}

int es_qplan_destroy(es_qplan_t* plan) {
    if (plan == nullptr) return ES_OK;
    const int rc = release_device_memory(plan->device, plan->d_tab, plan->d_scratch,
                                         "es_qplan_destroy");
    delete plan;
    return rc;
}

uint64_t es_qplan_numel(const es_qplan_t* plan) { return plan ? plan->numel : 0; }

uint64_t es_qplan_device_bytes(const es_qplan_t* plan) {
    return plan ? sizeof(esq::DevQTensor) * (plan->n_tensors + 1) + kScratchBytes : 0;
}

int es_qperturb(es_qplan_t* plan, uint64_t seed, int32_t sign, float sigma, es_stream_t stream) {
    return qperturb_impl(plan, seed, sign, sigma, stream, QKind::kPerturb, "es_qperturb");
}

int es_qrestore(es_qplan_t* plan, uint64_t seed, int32_t sign, float sigma, es_stream_t stream) {
    return qperturb_impl(plan, seed, sign, sigma, stream, QKind::kRestore, "es_qrestore");
}

int es_qswap(es_qplan_t* plan, uint64_t seed_from, int32_t sign_from, float sigma_from,
             uint64_t seed_to, int32_t sign_to, float sigma_to, es_stream_t stream) {
    if (plan == nullptr) return fail(ES_ERR_INVALID_ARG, "es_qswap: null plan");
    if ((sign_from != 1 && sign_from != -1) || (sign_to != 1 && sign_to != -1))
        return fail(ES_ERR_INVALID_ARG, "es_qswap: signs must be +1 or -1");
    if (!std::isfinite(sigma_from) || sigma_from < 0.0f || !std::isfinite(sigma_to) ||
        sigma_to < 0.0f)
        return fail(ES_ERR_INVALID_ARG, "es_qswap: sigmas must be finite and >= 0");
    // es_qrestore(from) then es_qperturb(to); a zero sigma makes its half the
    // identity, as in those calls (its pass would still clamp codes)
    if (sigma_from == 0.0f)
        return qperturb_impl(plan, seed_to, sign_to, sigma_to, stream, QKind::kPerturb, "es_qswap");
    if (sigma_to == 0.0f)
        return qperturb_impl(plan, seed_from, sign_from, sigma_from, stream, QKind::kRestore,
                             "es_qswap");
    const int rc = check_qdevice(plan);
    if (rc != ES_OK) return rc;
    QPass ps = {};
    ps.m = qmember(seed_to, sign_to, sigma_to);
    ps.m_from = qmember(seed_from, sign_from, sigma_from);
    return launch_qpass(plan, QKind::kSwap, ps, static_cast<hipStream_t>(stream));
}

int es_qupdate(es_qplan_t* plan, const uint64_t* seeds, const int32_t* signs,
               const float* rewards_dev, uint32_t n_members, const es_update_opts_t* opts,
               float* z_out_dev, int32_t* status_out_dev, es_stream_t stream) try {
    if (plan == nullptr) return fail(ES_ERR_INVALID_ARG, "es_qupdate: null plan");
    int rc = validate_update("es_qupdate", seeds, signs, rewards_dev, n_members, opts);
    if (rc != ES_OK) return rc;
    if (opts->flags & ES_UPDATE_MASTER)
        return fail(ES_ERR_INVALID_ARG, "es_qupdate: quantized plans have no binary32 masters");
    rc = check_qdevice(plan);
    if (rc == ES_OK)
        rc = check_update_arrays("es_qupdate", plan->device, rewards_dev, n_members, z_out_dev,
                                 status_out_dev);
    if (rc != ES_OK) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    rc = prepare_update(plan->d_scratch, seeds, signs, rewards_dev, n_members, opts, z_out_dev,
                        status_out_dev, s);
    if (rc != ES_OK) return rc;
    QPass ps = {};
    ps.dk0 = static_cast<uint32_t>(opts->round_seed);
    ps.dk1 = static_cast<uint32_t>(opts->round_seed >> 32);
    return launch_qpass(plan, QKind::kUpdate, ps, s);
} catch (const std::bad_alloc&) {
    return fail(ES_ERR_NOMEM, "es_qupdate: host allocation failed");
}

int es_stream_pass(es_plan_t* plan, es_stream_t stream) {
    if (plan == nullptr) return fail(ES_ERR_INVALID_ARG, "es_stream_pass: null plan");
    const int rc = check_device(plan);
    if (rc != ES_OK) return rc;
    Segment seg[2];
    const int n_seg = plan_segments(plan, seg);
    for (int k = 0; k < n_seg; ++k) {
        const Segment& g = seg[k];
        hipLaunchKernelGGL(stream_kernel(plan->threads, plan->groups), dim3(g.grid_perturb),
                           dim3(plan->threads), 0, static_cast<hipStream_t>(stream), g.tiles,
                           g.n_full, g.n_tail, 0u);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(e, "es_stream_kernel launch");
    }
    return ES_OK;
}

int es_hbm_calibrate(void* buf_dev, uint64_t bytes, int32_t mode, uint32_t* sink_dev,
                     es_stream_t stream) {
    constexpr uint64_t kTileBytes = uint64_t(kDefaultThreads) * kDefaultGroups * 16;
    const int32_t kind = mode & ~ES_CALIBRATE_TEMPORAL;
    const bool nt = (mode & ES_CALIBRATE_TEMPORAL) == 0;
    if (mode < 0 || kind > 2)
        return fail(ES_ERR_INVALID_ARG,
                    "es_hbm_calibrate: mode not 0, 1 or 2 (optionally | ES_CALIBRATE_TEMPORAL)");
    if (buf_dev == nullptr || (kind == 0 && sink_dev == nullptr))
        return fail(ES_ERR_INVALID_ARG, "es_hbm_calibrate: null pointer");
    if (bytes == 0 || bytes % kTileBytes != 0)
        return fail(ES_ERR_INVALID_ARG, "es_hbm_calibrate: bytes not a positive multiple of 131072");
    if (reinterpret_cast<uintptr_t>(buf_dev) % 16 != 0 ||
        (kind == 0 && reinterpret_cast<uintptr_t>(sink_dev) % 4 != 0))
        return fail(ES_ERR_ALIGN, "es_hbm_calibrate: buffer not 16-byte aligned");
    int device = -1;
    int rc = current_device(&device);
    if (rc == ES_OK) rc = check_access(buf_dev, bytes, device, "es_hbm_calibrate: buffer");
    if (rc == ES_OK && kind == 0)
        rc = check_access(sink_dev, 4, device, "es_hbm_calibrate: sink");
    if (rc != ES_OK) return rc;
    int cus = 0;
    hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
    const uint64_t n_tiles = bytes / kTileBytes;
    const dim3 grid(static_cast<uint32_t>(std::min<uint64_t>(n_tiles, uint64_t(cus))));
    const hipStream_t s = static_cast<hipStream_t>(stream);
    u32x4_t* buf = static_cast<u32x4_t*>(buf_dev);
    using CalKernel = void (*)(u32x4_t*, uint64_t, uint32_t*, uint32_t);
    constexpr int kT = kDefaultThreads, kG = kDefaultGroups;
    const CalKernel kernels[2][3] = {
        {es_calibrate_kernel<kT, kG, 0, false>, es_calibrate_kernel<kT, kG, 1, false>,
         es_calibrate_kernel<kT, kG, 2, false>},
        {es_calibrate_kernel<kT, kG, 0, true>, es_calibrate_kernel<kT, kG, 1, true>,
         es_calibrate_kernel<kT, kG, 2, true>}};
    hipLaunchKernelGGL(kernels[nt ? 1 : 0][kind], grid, dim3(kDefaultThreads), 0, s, buf, n_tiles,
                       sink_dev, 0u);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "es_calibrate_kernel launch");
    return ES_OK;
}

int es_plan_checksum(es_plan_t* plan, uint64_t* out_dev, es_stream_t stream) {
    if (plan == nullptr || out_dev == nullptr)
        return fail(ES_ERR_INVALID_ARG, "es_plan_checksum: null pointer");
    if (reinterpret_cast<uintptr_t>(out_dev) % 8 != 0)
        return fail(ES_ERR_ALIGN, "es_plan_checksum: output not 8-byte aligned");
    int rc = check_device(plan);
    if (rc == ES_OK) rc = check_access(out_dev, 8, plan->device, "es_plan_checksum: output");
    if (rc != ES_OK) return rc;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    unsigned long long* out = reinterpret_cast<unsigned long long*>(out_dev);
    hipLaunchKernelGGL(es_zero_u64_kernel, dim3(1), dim3(64), 0, s, out);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "es_zero_u64_kernel launch");
    Segment seg[2];
    const int n_seg = plan_segments(plan, seg);
    for (int k = 0; k < n_seg; ++k) {
        const Segment& g = seg[k];
        hipLaunchKernelGGL(checksum_kernel(plan->threads, plan->groups, g.rows != nullptr),
                           dim3(g.grid_update), dim3(plan->threads), 0, s, g.tiles, g.n_full,
                           g.n_tail, g.rows, out);
        e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(e, "es_checksum_kernel launch");
    }
    return ES_OK;
}

int es_qplan_checksum(es_qplan_t* plan, uint64_t* out_dev, es_stream_t stream) {
    if (plan == nullptr || out_dev == nullptr)
        return fail(ES_ERR_INVALID_ARG, "es_qplan_checksum: null pointer");
    if (reinterpret_cast<uintptr_t>(out_dev) % 8 != 0)
        return fail(ES_ERR_ALIGN, "es_qplan_checksum: output not 8-byte aligned");
    int rc = check_qdevice(plan);
    if (rc == ES_OK) rc = check_access(out_dev, 8, plan->device, "es_qplan_checksum: output");
    if (rc != ES_OK) return rc;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    unsigned long long* out = reinterpret_cast<unsigned long long*>(out_dev);
    hipLaunchKernelGGL(es_zero_u64_kernel, dim3(1), dim3(64), 0, s, out);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "es_zero_u64_kernel launch");
    if (plan->n_full + plan->n_tail == 0) return ES_OK;
    hipLaunchKernelGGL(qchecksum_kernel(plan->threads, plan->groups), dim3(plan->grid),
                       dim3(plan->threads), 0, s, plan->d_tab, plan->n_full, plan->n_tail, out);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "es_qchecksum_kernel launch");
    return ES_OK;
}

double es_sigma_cosine(double sigma0, double sigma_T, uint32_t t, uint32_t T) {
    if (T == 0 || t > T) return NAN;
    return sigma_T + (sigma0 - sigma_T) * (1.0 + std::cos(M_PI * double(t) / double(T))) / 2.0;
}

int es_philox_words(uint64_t seed, uint32_t tensor_id, uint32_t domain, uint64_t quad0,
                    uint64_t n_quads, uint32_t* out_dev, es_stream_t stream) {
    if (out_dev == nullptr) return fail(ES_ERR_INVALID_ARG, "es_philox_words: null output");
    if (n_quads > (uint64_t(1) << 28)) return fail(ES_ERR_INVALID_ARG, "es_philox_words: n_quads too large");
    if (reinterpret_cast<uintptr_t>(out_dev) % 16 != 0)
        return fail(ES_ERR_ALIGN, "es_philox_words: output not 16-byte aligned");
    if (n_quads == 0) return ES_OK;
    int device = -1;
    int rc = current_device(&device);
    if (rc == ES_OK) rc = check_access(out_dev, 16 * n_quads, device, "es_philox_words: output");
    if (rc != ES_OK) return rc;
    const uint32_t blocks = static_cast<uint32_t>((n_quads + kAuxBlock - 1) / kAuxBlock);
    hipLaunchKernelGGL(es_philox_words_kernel, dim3(blocks), dim3(kAuxBlock), 0,
                       static_cast<hipStream_t>(stream), static_cast<uint32_t>(seed),
                       static_cast<uint32_t>(seed >> 32), tensor_id, domain, quad0, n_quads,
                       reinterpret_cast<uint4*>(out_dev));
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "es_philox_words_kernel launch");
    return ES_OK;
}

int es_normals(uint64_t seed, uint32_t tensor_id, uint64_t elem0, uint64_t n, float* out_dev,
               es_stream_t stream) {
    if (out_dev == nullptr) return fail(ES_ERR_INVALID_ARG, "es_normals: null output");
    if (n > (uint64_t(1) << 30)) return fail(ES_ERR_INVALID_ARG, "es_normals: n too large");
    if (elem0 > (uint64_t(1) << 62) - n) return fail(ES_ERR_INVALID_ARG, "es_normals: element range beyond 2^62");
    if (n == 0) return ES_OK;
    int device = -1;
    int rc = current_device(&device);
    if (rc == ES_OK) rc = check_access(out_dev, 4 * n, device, "es_normals: output");
    if (rc != ES_OK) return rc;
    const uint64_t quads = ((elem0 + n - 1) >> 2) - (elem0 >> 2) + 1;
    const uint32_t blocks = static_cast<uint32_t>((quads + kAuxBlock - 1) / kAuxBlock);
    hipLaunchKernelGGL(es_normals_kernel, dim3(blocks), dim3(kAuxBlock), 0,
                       static_cast<hipStream_t>(stream), static_cast<uint32_t>(seed),
                       static_cast<uint32_t>(seed >> 32), tensor_id, elem0, n, out_dev);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "es_normals_kernel launch");
    return ES_OK;
}

int es_tile_layout(uint64_t addr, uint64_t numel, uint32_t offset8, es_tile_info_t* out,
                   uint64_t cap, uint64_t* n_tiles) try {
    if (n_tiles == nullptr) return fail(ES_ERR_INVALID_ARG, "es_tile_layout: null n_tiles");
    *n_tiles = 0;
    if (numel > (uint64_t(1) << 60) - 8 * uint64_t(offset8))
        return fail(ES_ERR_INVALID_ARG, "es_tile_layout: 8 * offset8 + numel above 2^60");
    if (cap > 0 && out == nullptr) return fail(ES_ERR_INVALID_ARG, "es_tile_layout: null output");
    if (numel > 0 && (addr & 1u)) return fail(ES_ERR_ALIGN, "es_tile_layout: address not 2-byte aligned");
    int threads = 0, groups = 0;
    launch_shape(threads, groups);
    const uint64_t tile_elems = uint64_t(threads) * groups * kGroupElems;
    if (numel / tile_elems > kMaxLayoutTiles)
        return fail(ES_ERR_INVALID_ARG, "es_tile_layout: more than 2^22 tiles");
    std::vector<DevTile> full, tail;
    tile_tensor(reinterpret_cast<uint16_t*>(static_cast<uintptr_t>(addr)), numel,
                8 * uint64_t(offset8), 0u, tile_elems, full, tail);
    const uint64_t n = full.size() + tail.size();
    for (uint64_t i = 0; i < std::min(cap, n); ++i) {
        const DevTile& d = i < full.size() ? full[i] : tail[i - full.size()];
        out[i] = es_tile_info_t{d.elem0, d.limit, i < full.size() ? 1u : 0u, d.aligned16};
    }
    *n_tiles = n;
    return ES_OK;
} catch (const std::bad_alloc&) {
    return fail(ES_ERR_NOMEM, "es_tile_layout: host allocation failed");
}

const char* es_strerror(int code) {
    switch (code) {
        case ES_OK: return "ES_OK";
        case ES_ERR_INVALID_ARG: return "ES_ERR_INVALID_ARG";
        case ES_ERR_ALIGN: return "ES_ERR_ALIGN";
        case ES_ERR_HIP: return "ES_ERR_HIP";
        case ES_ERR_DEVICE: return "ES_ERR_DEVICE";
        case ES_ERR_NOMEM: return "ES_ERR_NOMEM";
        default: return "ES_ERR_UNKNOWN";
    }
}

const char* es_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
