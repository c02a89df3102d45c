/*
 * esopt.h -- C ABI of the MI355X (gfx950) ES parameter-path library.
 *
 * What it computes (arXiv 2608.17310, "Agentic ESOpt"):
 *   Section 3 samples G full-parameter Gaussian directions eps_i around the
 *   current parameters theta, evaluates each perturbed model theta + sigma
 *   eps_i, z-scores the rewards within the population and applies
 *   theta <- theta + (alpha / G) sum_i zhat_i eps_i.  Only the integer seed
 *   of each direction is stored; the perturbation is applied and reverted in
 *   place, and the direction is regenerated from its seed for the update
 *   (Section 3; Appendix D.6).  Section 3.1 decays sigma on a cosine
 *   schedule.  Appendix C.1 gives the canonical estimator with 1/(G sigma).
 *
 * Noise definition (the paper names no generator; this is the library's):
 *   eps_j of element j of the tensor with noise identity `tensor_id`, for a
 *   64-bit seed, comes from Philox4x32-10 (Salmon et al., SC'11) with
 *     key     = (seed & 0xffffffff, seed >> 32)
 *     counter = (q & 0xffffffff, q >> 32, tensor_id, 0),  q = j >> 2
 *   Word pair (w0,w1) serves elements 4q, 4q+1 and (w2,w3) serves 4q+2,
 *   4q+3.  With m(w) = w & (2^23 - 1): radius uniform u = (m(wa) + 0.5)
 *   * 2^-23, angle v = m(wb) * 2^-23 turns; Box-Muller (1958):
 *   r = sqrt(-2 ln u), phi = 2 pi v; first element r cos(phi), second
 *   r sin(phi).  The GPU evaluates this in binary32.
 *
 * Parameters are bf16 (the paper states no dtype; its memory figures imply
 * 16-bit weights).  Each result is computed in binary32 and rounded to bf16
 * round-to-nearest-even (the update can instead round stochastically), with
 * exactly one read and one write per element.  Int8 and fp8 (E4M3)
 * parameters with per-row scales have a plan of their own (es_qplan_*,
 * further down).
 *
 * Conventions for every call:
 *   - Device pointers are HIP device memory of the device current at the
 *     call; the caller owns every buffer it passes.  A plan keeps the
 *     tensors' addresses, so they must stay allocated and unmoved while the
 *     plan exists; calls on one plan must be ordered (one stream, or
 *     externally synchronised) because they share the plan's small scratch.
 *   - `stream` is a hipStream_t (NULL: the default stream).  Every call is
 *     stream-ordered and returns without synchronising the host; launch
 *     errors are reported by the return code.  The passes (perturb, restore,
 *     swap, update, z-score and their quantized counterparts) only launch kernels
 *     on `stream` -- no memset, no host synchronisation, host arrays copied
 *     into kernel arguments -- so they can be captured into a HIP graph; a
 *     replay repeats the captured arguments (seeds, signs, sigma, alpha).
 *   - Every device pointer a call receives (tensors and scales at plan
 *     creation, rewards / z / status arrays and hook outputs per call) is
 *     checked with the runtime before any launch: it must be device or
 *     managed memory of the current device with the whole range inside one
 *     allocation, or mapped pinned host memory; otherwise the call fails
 *     with ES_ERR_INVALID_ARG.  (A plan's tensors are checked once, when it
 *     is created.)
 *   - Return value: ES_OK (0) or a negative ES_ERR_* code; es_strerror()
 *     names a code, es_last_error() gives the detail of the last failure on
 *     the calling thread.  A call that fails validation launches nothing and
 *     leaves every buffer untouched.
 */
#ifndef ESOPT_H
#define ESOPT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ES_OK                0
#define ES_ERR_INVALID_ARG  -1   /* null pointer, bad size, sign, sigma, flags */
#define ES_ERR_ALIGN        -2   /* bf16 data not 2-byte aligned, scales not 4-byte aligned */
#define ES_ERR_HIP          -3   /* a HIP runtime call or launch failed */
#define ES_ERR_DEVICE       -4   /* current device differs from the plan's */
#define ES_ERR_NOMEM        -5   /* device or host allocation failed */

#define ES_MAX_MEMBERS      1024u   /* population size limit of es_update */
#define ES_MAX_TENSORS      (1u << 20)

/* es_update flags */
#define ES_UPDATE_DIV_SIGMA     1u  /* c = alpha / (G sigma) (Appendix C.1)
                                       instead of the paper's alpha / G */
#define ES_REWARDS_ARE_WEIGHTS  2u  /* use rewards as zhat directly (no z-score) */
#define ES_UPDATE_STOCHASTIC_ROUND 4u /* round the update stochastically (round_seed) */
#define ES_UPDATE_MASTER        8u  /* update the plan's binary32 masters and rewrite
                                       the bf16 values from them (es_plan_set_master) */

typedef void* es_stream_t;          /* hipStream_t */

/* One parameter tensor: `numel` contiguous bf16 values at device address
 * `data` (2-byte aligned; 16-byte alignment takes the vector path).
 * `tensor_id` is the tensor's noise identity (counter word 2) and must be
 * unique within a plan and stable across calls; the list index is the usual
 * choice.  numel may be 0 (the tensor is skipped).
 * `offset8` places a shard: element i of `data` carries the noise of element
 * 8 * offset8 + i of the whole tensor `tensor_id`, so a shard holding a
 * contiguous range of a tensor (a row-parallel slice, a flat-parameter
 * shard) regenerates exactly the whole tensor's noise there, with no
 * communication.  0 for a tensor that is not sharded. */
typedef struct es_tensor {
    void*    data;
    uint64_t numel;
    uint32_t tensor_id;
    uint32_t offset8;
} es_tensor_t;

/* Opaque plan: the tensor list laid out as tiles for one launch per pass,
 * plus O(ES_MAX_MEMBERS) device scratch for the update's member table. */
typedef struct es_plan es_plan_t;

/* Build a plan over `n_tensors` tensors (1 .. ES_MAX_TENSORS) on the current
 * device.  Copies the list; does not touch the tensors' values.  Errors:
 * INVALID_ARG for a null pointer, n_tensors out of range, duplicate
 * tensor_id, null data with numel > 0, 8 * offset8 + numel above 2^60, or
 * tensors whose byte ranges overlap; ALIGN for odd addresses; NOMEM / HIP for
 * allocation failures.  On success *out owns 32 bytes of device memory per
 * tile of 65 536 elements (0.024 % of the parameter bytes; see
 * es_tile_layout) and ~42 KB of scratch, freed by es_plan_destroy;
 * es_plan_device_bytes reports the total. */
int es_plan_create(const es_tensor_t* tensors, uint32_t n_tensors, es_plan_t** out);

/* A rectangular block of a row-major bf16 tensor, as one GPU holds it under
 * tensor parallelism when the split runs across columns (a row-parallel
 * layer's weight: a range of every row): `rows` x `cols` values stored
 * contiguously at `data` (block row i at data + i * cols elements), which are
 * the whole tensor's elements (row0 + i) * row_len + col0 + j, i < rows,
 * j < cols.  Each carries the noise of that whole-tensor index (Section 3:
 * the noise is regenerated from the seed and the element's place), so every
 * pass over the block leaves exactly the values the same pass over the whole
 * tensor leaves there, and block checksums add up to the whole tensor's.
 * Requirements: col0 + cols <= row_len; the first index row0 * row_len + col0
 * is a multiple of 8; a block that is not one contiguous range of the tensor
 * (rows > 1 and cols < row_len) also has cols and row_len multiples of 8
 * (every hidden and intermediate size of the paper's models is); every index
 * is below 2^60.  A whole tensor is {data, 1, numel, numel, 0, 0}; an
 * es_tensor_t shard is {data, 1, numel, its tensor's numel, 0, 8 * offset8}.
 * rows * cols may be 0 (the block is skipped). */
typedef struct es_block {
    void*    data;
    uint64_t rows;
    uint64_t cols;
    uint64_t row_len;       /* the whole tensor's row length */
    uint64_t row0;          /* the block's first row in the whole tensor */
    uint64_t col0;          /* the block's first column in the whole tensor */
    uint32_t tensor_id;     /* as in es_tensor_t: unique within a plan */
    uint32_t reserved;      /* must be 0 */
} es_block_t;

/* es_plan_create over blocks (Section 3, the same passes: es_perturb,
 * es_restore, es_swap, es_update, es_update_noalloc, es_plan_checksum and
 * es_stream_pass accept the plan).  Blocks that are one contiguous range of
 * their tensor are laid out exactly as es_plan_create lays out tensors and
 * shards; the others are cut into pieces of whole rows (under 2^31 elements
 * each) whose tiles carry the piece's row map, and the passes run over them
 * in a second launch.  Errors: as es_plan_create (n_blocks for n_tensors),
 * plus INVALID_ARG for a block that breaks a requirement above or has
 * reserved != 0, and for rows * cols above 2^60. */
int es_plan_create_blocks(const es_block_t* blocks, uint32_t n_blocks, es_plan_t** out);

/* Free a plan (NULL is a no-op).  Synchronises the plan's device first (made
 * current for the call; the caller's current device is restored) so that no
 * queued launch still reads the plan's tables.  The plan is freed even when a
 * step fails; the first failure is returned. */
int es_plan_destroy(es_plan_t* plan);

/* Total number of bf16 elements and number of tiles of a plan. */
uint64_t es_plan_numel(const es_plan_t* plan);
uint64_t es_plan_tiles(const es_plan_t* plan);

/* Device memory a plan allocates for itself (its tile descriptors and
 * member scratch), in bytes: everything the method needs beyond the parameters
 * (Section 3: memory stays at inference level).  0 for NULL. */
uint64_t es_plan_device_bytes(const es_plan_t* plan);

/* Perturb in place (Section 3; Appendix D.6):
 *   theta_j <- RNE_bf16(theta_j + sign * sigma * eps_j(seed))
 * for every element of every tensor of the plan, one kernel launch.
 * sign is +1 or -1 (antithetic member); sigma is finite and >= 0; sigma == 0
 * leaves theta bit-for-bit unchanged and launches nothing. */
int es_perturb(es_plan_t* plan, uint64_t seed, int32_t sign, float sigma, es_stream_t stream);

/* Revert a perturbation (Section 3; Appendix D.6): es_perturb with -sign,
 *   theta_j <- RNE_bf16(theta_j - sign * sigma * eps_j(seed)).
 * Because each step rounds to bf16, the round trip returns theta except for
 * rounding residues (about 5% of N(0,0.02) elements move by one ulp at
 * sigma = 1e-3). */
int es_restore(es_plan_t* plan, uint64_t seed, int32_t sign, float sigma, es_stream_t stream);

/* Move the perturbation from one member to the next in one pass (Section 3;
 * Appendix D.6 -- revert member a after its evaluation, apply member b):
 *   mid_j   = RNE_bf16(theta_j - sign_from sigma_from eps_j(seed_from))
 *   theta_j <- RNE_bf16(mid_j + sign_to sigma_to eps_j(seed_to))
 * with one read and one write per element, both noise streams generated in
 * registers and the intermediate rounded in registers: the result is bit for
 * bit that of es_restore(from) followed by es_perturb(to), at half the
 * memory traffic.  Rounding the intermediate keeps a walk over many members
 * anchored to the starting parameters (a revert that stays in the value's
 * binade lands exactly on it), where a single rounding of
 * theta - a + b would accumulate each member's rounding error.  The same
 * seed on both sides (an antithetic partner) generates its noise once.  A
 * zero sigma makes its half the identity; both zero launches nothing.
 * Signs +1 or -1; sigmas finite and >= 0. */
int es_swap(es_plan_t* plan, uint64_t seed_from, int32_t sign_from, float sigma_from,
            uint64_t seed_to, int32_t sign_to, float sigma_to, es_stream_t stream);

/* Population z-score (Section 3): mu = mean(R), s = sqrt(mean((R - mu)^2)),
 *   z_i = (R_i - mu) / (s + eps),
 * computed in fp64 by one wavefront and written as binary32 to z_dev[n].
 * All rewards equal (including n == 1) gives z = 0 exactly.  If any reward is
 * not finite, z = 0 and *status_dev = 1, else *status_dev = 0 (status_dev may
 * be NULL).  rewards_dev and z_dev: device arrays of n floats, 1 <= n <=
 * ES_MAX_MEMBERS; they may alias.  eps must be finite and >= 0. */
int es_zscore(const float* rewards_dev, uint32_t n, float eps, float* z_dev,
              int32_t* status_dev, es_stream_t stream);

typedef struct es_update_opts {
    float    alpha;       /* step size, finite */
    float    sigma;       /* sigma_t of this generation; read only with
                             ES_UPDATE_DIV_SIGMA (then finite and > 0) */
    float    zscore_eps;  /* epsilon of the z-score denominator, >= 0 (1e-8) */
    uint32_t flags;       /* ES_UPDATE_DIV_SIGMA | ES_REWARDS_ARE_WEIGHTS |
                             ES_UPDATE_STOCHASTIC_ROUND | ES_UPDATE_MASTER */
    uint64_t round_seed;  /* key of the stochastic-rounding draws; read only
                             with ES_UPDATE_STOCHASTIC_ROUND */
} es_update_opts_t;

/* Fused reward-weighted update (Section 3; Appendix C.1 with
 * ES_UPDATE_DIV_SIGMA):
 *   zhat = zscore(rewards) (or rewards as given with ES_REWARDS_ARE_WEIGHTS)
 *   c    = alpha / G  (or alpha / (G sigma)),  G = n_members
 *   w_d  = sum over members i with seed d of c * sign_i * zhat_i   (fp64)
 *   theta_j <- RNE_bf16(theta_j + sum_d w_d eps_j(seed_d))
 * Members sharing a seed (antithetic pairs) are merged into one weight, so
 * the noise of each distinct seed is generated once per element; the sum is
 * accumulated in binary32 registers and theta is read and written once.
 * Seeds with a zero merged weight are skipped, and when no weight is nonzero
 * theta is not written at all.
 * The paper does not state how updates are rounded.  With
 * ES_UPDATE_STOCHASTIC_ROUND, instead of RNE: x = theta_j + sum (binary32),
 * and x moves from its truncation toward zero on the bf16 grid one step away
 * from zero when r_j >= 2^16 - (low 16 bits of x), r_j a 16-bit draw; so the
 * expected result is x.  Draws: key = (round_seed lo, hi), one Philox4x32-10
 * call at counter (g lo, g hi, tensor_id, 1), g = j >> 3, serves elements
 * 8g..8g+7; element j takes word (j & 7) >> 1, low half for even j, high
 * half for odd j.  Overflow past the largest finite bf16 gives infinity; NaN
 * gives 0x7FC0.  A non-finite reward leaves theta unchanged
 * and sets the status word to 1.
 * With ES_UPDATE_MASTER (a plan with masters, es_plan_set_master; not with
 * ES_UPDATE_STOCHASTIC_ROUND): the sum is added to the binary32 master m_j
 * instead, m_j <- m_j + sum (one binary32 rounding of the binary32 sum), and
 * every bf16 value is rewritten as RNE_bf16(m_j) without being read -- also
 * when the update adds nothing (then the masters are not written), so the
 * bf16 values left by the generation's perturbations and reverts do not
 * matter and the last member need not be reverted.
 *   seeds, signs : host arrays of n_members entries (signs +1 or -1)
 *   rewards_dev  : device array of n_members binary32 rewards
 *   n_members    : 1 .. ES_MAX_MEMBERS
 *   z_out_dev    : optional device array of n_members floats receiving zhat
 *   status_out_dev: optional device int32 receiving the status word
 * The host arrays are read before the call returns. */
int es_update(es_plan_t* plan, const uint64_t* seeds, const int32_t* signs,
              const float* rewards_dev, uint32_t n_members,
              const es_update_opts_t* opts, float* z_out_dev,
              int32_t* status_out_dev, es_stream_t stream);

/* The last member's revert and the update in one pass (Section 3; Appendix
 * D.6: after the last member is evaluated its perturbation is reverted, then
 * the update regenerates every member's noise).  The same bits as
 *   es_restore(plan, restore_seed, restore_sign, restore_sigma, stream);
 *   es_update(plan, seeds, signs, rewards_dev, n_members, opts, z_out_dev,
 *             status_out_dev, stream);
 * theta is read and written once instead of twice: the restored member's
 * noise is generated once per element for both (its seed must be one of
 * `seeds`, else INVALID_ARG), the revert is rounded to bf16 in registers
 * exactly as es_restore rounds it, and the update is added to the result.
 * When the update adds nothing (no nonzero weight, or a non-finite reward:
 * status word 1) the reverted values are stored, as the two calls would
 * leave them.  restore_sign is +1 or -1, restore_sigma finite and >= 0
 * (0: the call is es_update).  Other arguments and errors as es_update. */
int es_restore_update(es_plan_t* plan, uint64_t restore_seed, int32_t restore_sign,
                      float restore_sigma, const uint64_t* seeds, const int32_t* signs,
                      const float* rewards_dev, uint32_t n_members,
                      const es_update_opts_t* opts, float* z_out_dev,
                      int32_t* status_out_dev, es_stream_t stream);

/* Binary32 master copies of a plan's parameters (an update-numerics variant
 * of Section 3's update, the library's: the update accumulates in binary32
 * and the bf16 parameters the rollouts read are its nearest-even rounding, so
 * updates far below a bf16 step are kept and no restore drift carries over
 * from one generation to the next).  masters[i] is the binary32 copy of the
 * plan's tensor (or block) i, in the same element order: numel (rows * cols)
 * floats, 16-byte aligned, device memory of the plan's device, overlapping
 * no other master and no bf16 tensor of the plan; the caller owns it and
 * keeps it in place while attached.  Used by es_update / es_update_noalloc
 * with ES_UPDATE_MASTER; the perturbation passes work on the bf16 values as
 * before.  Allocates 8 bytes per tile of device memory (es_plan_device_bytes
 * counts it); a second call replaces the masters, masters == NULL detaches
 * them (synchronising the plan's device first).  Errors: INVALID_ARG for a
 * count other than the plan's tensor count, a null master, one outside its
 * device's memory, or overlaps; ALIGN for a master not 16-byte aligned;
 * DEVICE, NOMEM, HIP as elsewhere. */
int es_plan_set_master(es_plan_t* plan, void* const* masters, uint32_t n);

/* Apply one member from the masters: every bf16 value becomes
 * RNE_bf16(m_j + sign sigma eps_j(seed)), m_j + sign sigma eps_j formed in
 * binary32 with one rounding, read from the plan's masters (which stay
 * unchanged) and written to the bf16 tensors without reading them (6 bytes
 * per parameter).  In a generation over a plan with masters it replaces
 * perturb, swap and restore: each candidate is applied afresh, so no revert
 * is needed and the weights a candidate is evaluated at do not depend on the
 * candidates before it (Section 3's theta + sigma eps_i, rounded once).
 * For bf16-representable masters the result is es_perturb's of those
 * values, bit for bit.  sigma 0 writes RNE_bf16(m_j) (the bf16 copy
 * refreshed from the masters; -0 stays -0) and uses the plan's scratch, as
 * es_update; sigma > 0 uses no scratch (one kernel launch per part of the
 * plan, which a HIP graph can capture).  Errors: INVALID_ARG (null plan, a
 * plan without masters, sign, sigma), DEVICE, HIP. */
int es_perturb_master(es_plan_t* plan, uint64_t seed, int32_t sign, float sigma,
                      es_stream_t stream);

/* es_update for callers that cannot allocate (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * arguments, checks, results and errors as es_update, bit for bit, but the
 * member tables, merged weights and header of the update live in a static
 * device array of 41 216 bytes (room for ES_MAX_MEMBERS members) instead of
 * the plan's scratch, and a successful call allocates no device or host
 * memory (the member tables are built in fixed arrays on the calling
 * thread's stack, about 52 KB).  n_members above ES_MAX_MEMBERS is refused
 * with ES_ERR_INVALID_ARG.  Each device holds its own copy of the array until
 * the process ends; the first call on a device looks up its address there
 * (with that device current) and keeps it.  Every call on one device shares
 * that array: calls that overlap on one GPU (on different streams, or from
 * different threads without ordering) race and give undefined results, so
 * order them like calls on one plan.  The array keeps the last call's
 * contents; nothing in it needs clearing, since each call writes every
 * entry it reads.  A failed call records its message with es_last_error
 * (formatting it may allocate host memory). */
int es_update_noalloc(es_plan_t* plan, const uint64_t* seeds, const int32_t* signs,
                      const float* rewards_dev, uint32_t n_members,
                      const es_update_opts_t* opts, float* z_out_dev,
                      int32_t* status_out_dev, es_stream_t stream);

/* 64-bit checksum of a plan's parameters, written to *out_dev (device
 * memory, 8-byte aligned):
 *   H = sum over elements of mix64(j K_J + tensor_id K_T + b K_B)  mod 2^64
 * with j the element's index in its whole tensor (shard offset included), b
 * its 16 bits, K_J = 0x9E3779B97F4A7C15, K_T = 0xC2B2AE3D27D4EB4F,
 * K_B = 0x165667B19E3779F9, and mix64 the finalizer of SplitMix64 (Steele,
 * Lea and Flood, OOPSLA 2014):
 *   z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27;
 *   z *= 0x94D049BB133111EB; z ^= z >> 31.
 * It serves the seed replay of Section 3 and Appendix D.6 (a run rebuilt from
 * its seed log can be checked against checksums recorded with it) and
 * replicas that must stay identical after each update.  The sum does not
 * depend on the launch shape, and the checksums of disjoint shards of a
 * tensor add up (mod 2^64) to the whole tensor's.  Reads the parameters once
 * (two launches: one clears *out_dev, one sums); an empty plan gives 0. */
int es_plan_checksum(es_plan_t* plan, uint64_t* out_dev, es_stream_t stream);

/* ---- int8 parameters (quantized ES; the paper lists it as future work,
 * Appendix A.2: scale-aware noise, stable updates, seed replay) ----
 *
 * A quantized tensor holds symmetric int8 codes q_j in [-127, 127] with
 * binary32 scales: theta_j = s_r q_j, r = j / row (row == 0: one scale for
 * the tensor).  Every pass moves codes by an integer offset k_j, the step d_j
 * in quanta rounded stochastically (E[k_j] = d_j), and clamps:
 * q_j <- clamp(q_j +- k_j, -127, 127) (so a code of -128 is clamped into the
 * range).  Elements whose scale is not a normal positive finite binary32
 * value are left unchanged, -128 included. */
typedef struct es_qtensor {
    void*        data;       /* device int8 codes, contiguous; any alignment
                                (16-byte aligned data takes the vector path) */
    const float* scales;     /* device binary32 scales, ceil(numel / row)
                                entries (1 when row == 0), 4-byte aligned */
    uint64_t     numel;      /* < 2^31 */
    uint32_t     row;        /* codes per scale: a multiple of 8, or 0 */
    uint32_t     tensor_id;  /* noise identity, unique within a plan */
} es_qtensor_t;

typedef struct es_qplan es_qplan_t;

/* Plan over int8 tensors (same ownership, device and launch-shape rules as
 * es_plan_create; overlapping code ranges and duplicate ids are rejected;
 * scales may be shared). */
int es_qplan_create(const es_qtensor_t* tensors, uint32_t n_tensors, es_qplan_t** out);

/* Code formats of a quantized plan (one format per plan). */
#define ES_QFORMAT_INT8  0u   /* symmetric int8 codes (above) */
#define ES_QFORMAT_E4M3  1u   /* fp8 E4M3 codes (below) */

/* A plan over fp8 E4M3 codes (format ES_QFORMAT_E4M3; ES_QFORMAT_INT8 is
 * es_qplan_create).  Each es_qtensor_t then holds one-byte codes of the OCP
 * 8-bit floating-point format with 4 exponent and 3 mantissa bits, bias 7
 * (PyTorch's float8_e4m3fn): theta_j = s_r v(c_j), v up to +-448, codes 0x7F
 * and 0xFF not a number; the scales, rows, ids and limits are as for int8.
 * The passes of the plan (es_qperturb, es_qrestore, es_qswap, es_qupdate,
 * es_qplan_checksum) then work on the E4M3 grid (Appendix A.2's quantized
 * ES, the library's reading): a pass forms x = v(c) + step, in scale units
 * and binary32, and rounds it onto the grid stochastically --
 *   lo = the largest grid value <= x, h the spacing to the next one,
 *   f = (x - lo) / h;  result = lo + h if f >= thr (perturb, update) or
 *   f > thr (restore), else lo;  clamped to [-448, 448]
 * -- with
 *   perturb: x = v + sign sigma eps_j / s, thr = 1 - u,
 *            u = (2 r + 1) 2^-10, r the top 9 bits of word j & 3 of element
 *            j's own noise call (as es_qperturb's int8 draw);
 *   restore: y = v - sign sigma eps_j / s, thr = u (the same u), which
 *            returns the original code exactly wherever the perturbation's
 *            x, the perturbed value and y stay in one binade of the grid, x
 *            below 448 (a perturbation into
 *            a coarser binade maps two codes to one, and its revert is off by
 *            at most one step of the coarser grid);
 *   update:  x = v + sum_d w_d eps_j(seed_d) / s with es_update's merged
 *            weights, thr = 1 - r 2^-16 with es_update's 16-bit stochastic
 *            rounding draws (domain 1 under opts->round_seed); always
 *            stochastic.
 * Not-a-number codes and the codes of invalid scales are left unchanged; a
 * zero result is +0 (code 0x00).  Errors as es_qplan_create, and
 * ES_ERR_INVALID_ARG for an unknown format. */
int es_qplan_create_format(const es_qtensor_t* tensors, uint32_t n_tensors, uint32_t format,
                           es_qplan_t** out);

/* A quantized plan over shards of tensors (the int8 and E4M3 counterpart of
 * es_tensor_t.offset8; Section 3: each element's noise is regenerated from
 * the seed and its place in its whole tensor, so a GPU holding a contiguous
 * range of a tensor needs no communication).  Code i of tensors[k] is code
 * elem0[k] + i of the whole tensor tensors[k].tensor_id: it takes that
 * code's noise, rounding draws (perturb and update) and checksum term, so
 * every pass over the shard leaves exactly the codes the same pass over the
 * whole tensor leaves there, and the checksums of disjoint shards add up
 * (mod 2^64) to the whole tensor's.  tensors[k].scales holds the shard's own
 * scales: scale r serves the shard's codes r row .. r row + row - 1 (the
 * whole tensor's scale elem0[k] / row + r); with row == 0 the one scale of
 * the tensor.  Requirements: elem0[k] a multiple of 16, and of row when
 * row > 0 (a shard starts on a row of scales); elem0[k] + numel below 2^31.
 * elem0 may be null (every shard starts at 0: es_qplan_create_format).
 * Errors as es_qplan_create_format, and ES_ERR_INVALID_ARG for an elem0 that
 * breaks a requirement. */
int es_qplan_create_shards(const es_qtensor_t* tensors, const uint64_t* elem0, uint32_t n_tensors,
                           uint32_t format, es_qplan_t** out);

/* A rectangular block of a row-major quantized tensor (the int8 / E4M3
 * counterpart of es_block_t, for column and row-and-column shards):
 * rows x cols one-byte codes stored contiguously at `data` (block row i at
 * data + i * cols), which are the whole tensor's codes
 * (row0 + i) * row_len + col0 + j, i < rows, j < cols.  Each takes the
 * noise, rounding draws and checksum term of that whole-tensor index
 * (Section 3), so every pass over the block leaves exactly the codes the
 * same pass over the whole tensor leaves there, and block checksums add up
 * to the whole tensor's.  `scales` and `row` describe the block's own codes
 * as in es_qtensor_t, in the block's storage order (scale r serves codes
 * r row .. r row + row - 1 of the block): a matrix with one scale per
 * row, split by columns, gives row = cols and the block's rows of scales;
 * one scale per g consecutive codes of a row (g dividing cols and col0)
 * gives row = g and the block's [rows, cols / g] scales.
 * Requirements: col0 + cols <= row_len; rows * cols below 2^31;
 * (row0 + rows - 1) * row_len + col0 + cols below 2^31; the first index
 * row0 * row_len + col0 a multiple of 16; a block that is not one
 * contiguous range of its tensor (rows > 1 and cols < row_len) also has
 * cols and row_len multiples of 16; row a multiple of 8, or 0.  rows * cols
 * may be 0 (the block is skipped). */
typedef struct es_qblock {
    void*        data;       /* device codes (any alignment, as es_qtensor_t) */
    const float* scales;     /* device binary32 scales of the block's codes */
    uint64_t     rows;
    uint64_t     cols;
    uint64_t     row_len;    /* codes per row of the whole tensor */
    uint64_t     row0;       /* the block's first row and column in it */
    uint64_t     col0;
    uint32_t     row;        /* codes per scale in the block's storage order */
    uint32_t     tensor_id;  /* noise identity, unique within a plan */
} es_qblock_t;

/* A quantized plan over blocks (format as es_qplan_create_format; blocks and
 * tensors share the passes, es_qplan_numel and es_qplan_checksum).  Errors as
 * es_qplan_create_format, and ES_ERR_INVALID_ARG for a block that breaks a
 * requirement above or overlaps another in memory. */
int es_qplan_create_blocks(const es_qblock_t* blocks, uint32_t n_blocks, uint32_t format,
                           es_qplan_t** out);
int es_qplan_destroy(es_qplan_t* plan);
uint64_t es_qplan_numel(const es_qplan_t* plan);
uint64_t es_qplan_device_bytes(const es_qplan_t* plan);   /* as es_plan_device_bytes */

/* Perturb (Section 3, in quanta): d_j = sign sigma eps_j(seed) / s_r with the
 * bf16 path's noise, k_j = floor(d_j + (2 r_j + 1) 2^-10) with r_j the top 9
 * bits of word j & 3 of element j's own noise call (bits the uniform map does
 * not read); q_j <- clamp(q_j + k_j).  es_qrestore regenerates the same k_j
 * and subtracts it, so perturb then restore returns every code whose
 * perturbed value was not clamped exactly.  sigma finite and >= 0 (0: nothing
 * runs). */
int es_qperturb(es_qplan_t* plan, uint64_t seed, int32_t sign, float sigma, es_stream_t stream);
int es_qrestore(es_qplan_t* plan, uint64_t seed, int32_t sign, float sigma, es_stream_t stream);

/* Revert one member and apply the next in one pass over the codes (the move
 * between candidates of Section 3 and Appendix D.6, as es_swap): exactly the
 * codes of es_qrestore(seed_from, sign_from, sigma_from) followed by
 * es_qperturb(seed_to, sign_to, sigma_to), both computed per code in
 * registers.  The passes are VALU-bound, so the fusion saves the second
 * pass's load, decode, pack and store (not its noise).  A zero sigma makes
 * its half the identity (the other half runs alone); both zero launches
 * nothing.  Signs +1 or -1; sigmas finite and >= 0. */
int es_qswap(es_qplan_t* plan, uint64_t seed_from, int32_t sign_from, float sigma_from,
             uint64_t seed_to, int32_t sign_to, float sigma_to, es_stream_t stream);

/* Update (Section 3 / Appendix C.1, in quanta): the z-score, coefficient and
 * merged weights of es_update, d_j = sum_d w_d eps_j(seed_d) / s_r,
 * k_j = floor(d_j + r_j 2^-16) with the 16-bit draws of es_update's
 * stochastic rounding (domain 1 under opts->round_seed); q_j <- clamp(q_j + k_j).  The rounding is
 * always stochastic (steps are usually a fraction of a quantum, which
 * rounding to nearest would drop); ES_UPDATE_STOCHASTIC_ROUND is accepted
 * and changes nothing.  Other arguments, status and z_out as es_update. */
int es_qupdate(es_qplan_t* plan, const uint64_t* seeds, const int32_t* signs,
               const float* rewards_dev, uint32_t n_members, const es_update_opts_t* opts,
               float* z_out_dev, int32_t* status_out_dev, es_stream_t stream);

/* Checksum of a quantized plan's codes (int8 or E4M3), as es_plan_checksum
 * with b the code's 8 bits (0 .. 255) and j its index in its tensor; the
 * scales are not included (no pass changes them). */
int es_qplan_checksum(es_qplan_t* plan, uint64_t* out_dev, es_stream_t stream);

/* Cosine schedule of the perturbation radius (Section 3.1):
 *   sigma_t = sigma_T + (sigma_0 - sigma_T) (1 + cos(pi t / T)) / 2,
 * 0 <= t <= T, T >= 1; returns NaN for arguments out of range.  Update t
 * (0-based) uses sigma_t. Host-only helper. */
double es_sigma_cosine(double sigma0, double sigma_T, uint32_t t, uint32_t T);

/* Calibration pass: reads every parameter of the plan and writes it back
 * unchanged, bit for bit, with the tiles, 16-byte nontemporal accesses and
 * launch shape of es_perturb but no arithmetic and no software pipelining
 * (each workgroup loads a whole tile, then stores it) -- the fastest
 * in-place stream over the plan's memory, so its duration is the practical
 * ceiling against which es_perturb's bandwidth is measured. */
int es_stream_pass(es_plan_t* plan, es_stream_t stream);

/* HBM calibration over a caller's flat device buffer of `bytes` bytes (a
 * positive multiple of 131072, 16-byte aligned), with the tile shape and
 * launch of es_perturb: 1024 lanes x 8 16-byte words per tile, one workgroup
 * per compute unit, nontemporal accesses (the passes' policy; with
 * ES_CALIBRATE_TEMPORAL or-ed into `mode`, ordinary loads and stores), each
 * tile loaded whole, then stored.  mode 0 reads every word (their XOR is folded into *sink_dev, a
 * device uint32, with one atomic per wave, so the reads are not dead code);
 * mode 1 writes every word (the buffer's contents become a pattern: the
 * 16-byte word of lane l in group u of tile t holds (t, u, l, 0)); mode 2
 * reads every word and writes it back unchanged.  With es_stream_pass these
 * give the practical read, write and in-place ceilings of the device's
 * memory against which the passes' bandwidth is read.  sink_dev is ignored
 * unless mode is 0. */
#define ES_CALIBRATE_TEMPORAL 4   /* es_hbm_calibrate: ordinary, not nontemporal, accesses */
int es_hbm_calibrate(void* buf_dev, uint64_t bytes, int32_t mode, uint32_t* sink_dev,
                     es_stream_t stream);

/* Test hooks exposing the device noise functions the kernels use.
 * es_philox_words: out_dev[4 i + k] = word k of the Philox call at counter
 *   (q & 0xffffffff, q >> 32, tensor_id, domain), q = quad0 + i,
 *   key from seed, for i < n_quads (n_quads <= 2^28).
 * es_normals: out_dev[i] = eps_j(seed) of element j = elem0 + i of tensor
 *   `tensor_id`, binary32, for i < n (n <= 2^30). */
int es_philox_words(uint64_t seed, uint32_t tensor_id, uint32_t domain,
                    uint64_t quad0, uint64_t n_quads, uint32_t* out_dev,
                    es_stream_t stream);
int es_normals(uint64_t seed, uint32_t tensor_id, uint64_t elem0, uint64_t n,
               float* out_dev, es_stream_t stream);

/* Test hook of the host-side tiling (no device access; the address is never
 * dereferenced): the tiles es_plan_create lays out for one bf16 tensor of
 * `numel` elements at address `addr` with shard offset `offset8`, with the
 * plan's launch shape.  Tile i covers elements [elem0, end) of the whole
 * tensor (8 * offset8 onwards); full tiles come first (full = 1:
 * tile-sized, starting where the address is a multiple of the tile's byte
 * size), then tail tiles.  Writes min(cap, count) entries to `out` (which
 * may be NULL when cap is 0) and the count to *n_tiles.  Errors: INVALID_ARG
 * for a null n_tiles, 8 * offset8 + numel > 2^60, or more than 2^22 tiles
 * (2^38 elements with the default tiles: the hook builds the whole list on
 * the host), ALIGN for an odd address. */
typedef struct es_tile_info {
    uint64_t elem0;
    uint64_t end;
    uint32_t full;
    uint32_t aligned16;
} es_tile_info_t;
int es_tile_layout(uint64_t addr, uint64_t numel, uint32_t offset8, es_tile_info_t* out,
                   uint64_t cap, uint64_t* n_tiles);

/* Static name of an error code; detail of the calling thread's last error. */
const char* es_strerror(int code);
const char* es_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ESOPT_H */
