/*
 * fiona.h -- C ABI of the MI355X (gfx950) hybrid weighted sum.
 *
 * The operation (Fiona, Sec. 4.2 "Exact Compilation of Routed Linear
 * Operators", Eq. (routed-example) and Eq. (shared-example)): a routed linear
 * layer computes every packed output ciphertext y_j from already prepared
 * (rotated) input ciphertexts A_i as
 *
 *     y_j = sum over raw terms (i, pi) of  pt_pi (*) A_i              (one PMult each)
 *         + sum over signed-sum uses (s, sigma, c) of  c * sigma * U_s
 *     U_s = sum over members (i, h) of  h * A_i,   h in {-1, 0, +1}   (Add / Sub / skip)
 *
 * where (*) is the slot-wise product, c is the reconstruction factor of the
 * group (applied once to the group's signed sum: "Grouping Reconstruction
 * Operations"), a signed sum U_s may be shared by several outputs, also with
 * all signs reversed (sigma = -1: "Sharing Signed Sums"), and the signed and
 * raw results of an output are added before any rescale ("Combining the
 * Signed and Raw Routes").  The library evaluates this exactly in every RNS
 * limb: ciphertexts are in the negacyclic NTT domain, where a PMult is an
 * element-wise product mod q_l and a constant factor c is a scalar product.
 * Rotation, key switching, rescale, encoding and bootstrapping are not part
 * of it.
 *
 * Data layout ("limb-major"), all uint64 residues:
 *   ciphertext i, polynomial p (0 = c0, 1 = c1), limb l, coefficient k is
 *   element ((i * 2 + p) * L + l) * N + k of a ciphertext array;
 *   plaintext pi, limb l, coefficient k is element (pi * L + l) * N + k.
 *
 * Every function returns FIONA_OK (0) or a negative fiona_status and never
 * throws or aborts.  All objects are created and destroyed by the caller.
 */
#ifndef FIONA_H
#define FIONA_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum fiona_status {
  FIONA_OK = 0,
  FIONA_ERR_ARG = -1,          /* null pointer, zero or inconsistent size */
  FIONA_ERR_PLAN = -2,         /* layer description inconsistent (index out of range, bad CSR) */
  FIONA_ERR_UNSUPPORTED = -3,  /* N, L or a modulus outside the supported range */
  FIONA_ERR_ALIGN = -4,        /* a device pointer is not 8-byte aligned (rotation keys: 16-byte) */
  FIONA_ERR_ALIAS = -5,        /* the output buffer overlaps an input buffer */
  FIONA_ERR_HIP = -6,          /* a HIP runtime call failed (device allocation, copy, launch) */
  FIONA_ERR_NOMEM = -7,        /* host allocation failed */
  FIONA_ERR_NODEVICE = -8,     /* the plan was created host-only and has no device image */
  FIONA_ERR_PRECONDITION = -9, /* an input breaks a precondition (checked only where documented) */
  FIONA_ERR_BOUNDS = -10       /* a replayed access falls outside its buffer (fiona_check_ntt_offsets) */
} fiona_status;

/* Limits checked by fiona_ctx_create. */
#define FIONA_MAX_N (1u << 20)
#define FIONA_MAX_L 64u
#define FIONA_MODULUS_BITS 50      /* every modulus satisfies 2^20 < q < 2^50 */
#define FIONA_SCALE_BITS 20        /* every integer scale c satisfies c < 2^20 */
#define FIONA_MAX_MEMBERS 48u      /* longer ternary groups are split into exact sub-sums */
#define FIONA_MAX_INPUTS 159u      /* input ciphertexts of one pass: a 64-coefficient tile of every
                                      input (16 B each) plus one zero row fill the 160 KiB LDS; a layer
                                      with more inputs runs in passes over input ranges */
#define FIONA_MAX_LAYER_INPUTS 65536u   /* input ciphertexts per layer */

typedef struct fiona_ctx fiona_ctx;
typedef struct fiona_plan fiona_plan;

/*
 * fiona_ctx_create: RNS parameters of the ciphertexts.
 *   N       coefficients per limb, 1 <= N <= FIONA_MAX_N (any N; CKKS uses a
 *           power of two, and the kernel handles a partial last tile);
 *   L       number of RNS limbs, 1 <= L <= FIONA_MAX_L;
 *   moduli  host array of L moduli, each 2^20 < q_l < 2^50 (so that every
 *           integer scale, < 2^20, is a canonical residue).  The element-wise
 *           path does not need them to be NTT-friendly primes; CKKS callers
 *           pass primes q = 1 (mod 2N).
 * Host-only: no device memory is touched.  On success *out owns a context
 * that fiona_ctx_destroy frees.  Errors: FIONA_ERR_ARG (null), FIONA_ERR_UNSUPPORTED.
 */
int fiona_ctx_create(uint32_t N, uint32_t L, const uint64_t *moduli, fiona_ctx **out);
void fiona_ctx_destroy(fiona_ctx *ctx);

/* Plan flags. */
#define FIONA_PLAN_NO_SHARING 1u   /* evaluate every group's signed sum on its own (no reuse) */
#define FIONA_PLAN_HOST_ONLY 2u    /* build and check the plan on the host; upload nothing */
#define FIONA_PLAN_NO_LDS_SUMS 4u  /* never keep shared signed sums resident in LDS */
#define FIONA_PLAN_NO_PARTIAL_SHARING 8u   /* share only whole signed sums, no common sub-sums */
#define FIONA_PLAN_PER_CONTRIBUTION 16u    /* no grouping: a scalar product per nonzero signed term
                                              (the first compilation of Sec. 6.2; implies NO_SHARING) */
#define FIONA_PLAN_NO_OUTPUT_BURSTS 32u    /* store each output as soon as it is finished instead of
                                              buffering a round of outputs in LDS and writing them together
                                              (the default when outputs are at least 2.5% of the bytes) */
#define FIONA_PLAN_CHECK_INPUTS 64u        /* a checking plan: it keeps the layer's signs, and every
                                              fiona_hybrid_linear call checks its inputs' preconditions on the
                                              host first (synchronously; see fiona_plan_check_inputs) */

/*
 * One routed layer, in the raw per-(output, term) form the offline compiler
 * emits (paper Sec. 2.2 "Execution Plan": fixed before any query).  Host
 * arrays, all read during fiona_plan_create only (the caller keeps ownership).
 *
 * Raw route, per output CSR:
 *   pm_off[n_out+1]        terms of output j are pm_off[j] .. pm_off[j+1]-1
 *   pm_input[n_pm]         input ciphertext of each raw term (< n_in)
 *   pm_pt[n_pm]            plaintext of each raw term (< n_pt)
 * Signed route, per output CSR over groups, per group CSR over members:
 *   grp_off[n_out+1]       groups of output j are grp_off[j] .. grp_off[j+1]-1
 *   grp_mem_off[n_group+1] members of group g are grp_mem_off[g] .. grp_mem_off[g+1]-1
 *   mem_input[n_member]    input ciphertext of each member (< n_in)
 *   mem_sign[n_member]     sign h in {-1, 0, +1} of each member: the same
 *                          values the caller later passes as ternary_groups
 *   grp_scale[n_group]     index into the scales array of each group (< n_scale)
 * n_group and n_member are grp_off[n_out] and grp_mem_off[n_group].
 * Plaintext table layout:
 *   pt_pitch               words from one plaintext to the next in pt_diags:
 *                          0 means L*N (packed rows), otherwise at least L*N
 *                          (FIONA_ERR_ARG if less).  Words between rows are
 *                          never read.  fiona_pt_pitch_hint gives a padded
 *                          pitch that spreads the rows over the HBM banks.
 */
typedef struct fiona_layer_desc {
  uint32_t n_in, n_out, n_pt, n_scale;
  const uint32_t *pm_off;
  const uint32_t *pm_input;
  const uint32_t *pm_pt;
  const uint32_t *grp_off;
  const uint32_t *grp_mem_off;
  const uint32_t *mem_input;
  const int8_t *mem_sign;
  const uint32_t *grp_scale;
  uint32_t flags;
  uint64_t pt_pitch;
} fiona_layer_desc;

/*
 * fiona_pt_pitch_hint: a plaintext pitch for fiona_layer_desc.pt_pitch (in
 * words) that keeps the rows streamed together by one launch off the same
 * HBM banks: L*N rounded up to a multiple of 64 words, plus 128 words.  With
 * packed rows (pitch L*N, a multiple of 2 MiB at N = 2^16) every plaintext's
 * slice of a tile lands at the same bank offset; the padding spreads them.
 * Returns 0 for a null ctx.
 */
uint64_t fiona_pt_pitch_hint(const fiona_ctx *ctx);

/*
 * fiona_plan_create: compile one layer for the GPU.
 *   - checks every index of desc (FIONA_ERR_PLAN on any inconsistency);
 *   - drops members whose sign is 0 and groups with no nonzero member: they
 *     contribute nothing (Sec. 3 Obs. 2, the skip; Sec. 4.2 "contributes nothing");
 *   - splits groups of more than FIONA_MAX_MEMBERS members into sub-sums with
 *     the same scale (exact, since c*(U1 + U2) = c*U1 + c*U2);
 *   - unless FIONA_PLAN_NO_SHARING, finds signed sums that are equal or
 *     exactly opposite (same inputs, same or all reversed signs) across the
 *     layer and computes each once (Sec. 4.2 "Sharing Signed Sums"); sums
 *     used more than once are kept resident in LDS per position tile;
 *   - unless FIONA_PLAN_NO_SHARING or FIONA_PLAN_NO_PARTIAL_SHARING, also
 *     shares signed terms common to several sums that only partly overlap
 *     (Sec. 4.2, the candidate search with its estimate k*m - m - k of the
 *     Add/Sub saved by a common term of m members reused k times): the most
 *     reused common pair (two inputs, or inputs and earlier common terms,
 *     with fixed relative sign) is taken while the estimate is positive,
 *     the reuse pays for forming it once per tile and LDS rows are left.
 *     Each common term is formed once per position tile and then enters
 *     every sum that contains it as a single member;
 *   - uploads the compiled metadata to the current HIP device (synchronous)
 *     unless FIONA_PLAN_HOST_ONLY.
 *   - a layer with more than FIONA_MAX_INPUTS inputs is compiled as passes
 *     over consecutive input ranges of at most 128 inputs each: a pass takes
 *     the raw terms and the group members whose input falls in its range (a
 *     group spanning several ranges becomes one sub-sum per range with the
 *     group's scale, exact since c*(U1 + U2) = c*U1 + c*U2); the first pass
 *     stores the outputs and each later pass adds its sums to them mod q_l,
 *     so the outputs are read and written once more per extra pass; a range
 *     that no term reads gets no pass;
 * The plan keeps a reference to ctx (which must outlive it).  Errors:
 * FIONA_ERR_ARG (also a pt_pitch below L*N), FIONA_ERR_PLAN, FIONA_ERR_UNSUPPORTED
 * (more than FIONA_MAX_LAYER_INPUTS inputs, or a plaintext table beyond 2^48 bytes), FIONA_ERR_NOMEM, FIONA_ERR_HIP.
 * The plan owns a small device
 * workspace (the members of its signed sums, reordered by sign on every call),
 * so one plan must not be used by two streams at the same time.
 */
int fiona_plan_create(const fiona_ctx *ctx, const fiona_layer_desc *desc, fiona_plan **out);
void fiona_plan_destroy(fiona_plan *plan);

/* Operation counts of a compiled plan (per position and polynomial, as the
 * paper counts CKKS operations per ciphertext in Sec. 4.2 and Sec. 6.2). */
typedef struct fiona_plan_stats_t {
  uint64_t ct_terms;               /* all (output, term) pairs, sign-0 members included */
  uint64_t n_pmult;                /* raw terms: one PMult each */
  uint64_t n_member;               /* signed terms (members), sign 0 included */
  uint64_t n_member_nonzero;       /* signed terms with h != 0 */
  uint64_t n_use;                  /* (output, signed sum) uses: one scalar product each */
  uint64_t n_sum_distinct;         /* distinct signed sums after sharing */
  uint64_t n_sum_resident;         /* shared sums kept in LDS, computed once per tile */
  uint64_t pmult_per_contribution; /* PMults if every signed term were applied on its own */
  uint64_t pmult_grouped;          /* PMults after grouping: raw terms + uses */
  uint64_t addsub_unshared;        /* Add/Sub to form every use's signed sum on its own */
  uint64_t addsub_shared;          /* Add/Sub with each distinct sum formed once */
  uint64_t addsub_partial;         /* Add/Sub after also sharing common partial sums:
                                      distinct sums plus the common terms themselves */
  uint32_t tile;                   /* coefficients per workgroup */
  uint32_t waves;                  /* wavefronts per workgroup */
  uint32_t lds_bytes;              /* LDS per workgroup */
  uint32_t grid;                   /* workgroups per launch */
  uint32_t split_outputs;          /* outputs split into segments over several wavefronts */
  uint32_t segment_slots;          /* LDS rows holding the segments' partial residues */
  uint32_t n_partial;              /* common partial sums, each formed once per tile in LDS */
  uint32_t partial_levels;         /* longest chain of common terms built from common terms */
  uint32_t output_rounds;          /* rounds of outputs per tile, each ending in one burst of stores */
  uint32_t output_buffer_rows;     /* LDS rows (outputs) buffered per round; 0 = stored directly */
  uint32_t input_passes;           /* launches (input ranges) per call: 1 up to FIONA_MAX_INPUTS inputs;
                                      with several, the counts above add up over the passes (a group
                                      split over passes counts one use per pass) and the launch shape is
                                      the widest pass's */
} fiona_plan_stats_t;

int fiona_plan_stats(const fiona_plan *plan, fiona_plan_stats_t *out);

/*
 * fiona_plan_check_inputs: the preconditions of fiona_hybrid_linear that a
 * checking plan (FIONA_PLAN_CHECK_INPUTS) enforces, tested on host copies of
 * the call's arrays (Sec. 2.2: the plan is fixed offline from the weights,
 * so the signs a call passes must be the signs the plan was compiled from):
 *   signs   host, [n_member] int8: must equal the layer description's mem_sign
 *   scales  host, [n_scale] uint64: each < 2^20
 *   in      host or NULL, [n_in][2][L][N] uint64: each < 2^50
 *   pt      host or NULL, [n_pt] rows at the plan's pitch: each word of a
 *           row's first L*N < 2^50
 * Returns FIONA_OK, FIONA_ERR_PRECONDITION (the first failing check), or
 * FIONA_ERR_ARG (a null plan or array with a nonzero size, or a plan made
 * without FIONA_PLAN_CHECK_INPUTS, which keeps no signs).  Host only; works
 * with a host-only plan.
 * A checking plan's fiona_hybrid_linear copies ternary_groups, scales,
 * in_cts and pt_diags back to the host (on its stream, then waits for it),
 * runs this check, and returns FIONA_ERR_PRECONDITION without launching
 * anything if it fails.  It is a debugging aid: it allocates host memory
 * and is as slow as copying every input.
 */
int fiona_plan_check_inputs(const fiona_plan *plan, const int8_t *signs, const uint64_t *scales, const uint64_t *in,
                            const uint64_t *pt);

/*
 * fiona_hybrid_linear: evaluate the layer (the hot path).
 *   in_cts          device, [n_in][2][L][N] uint64, every value < 2^50
 *                   (CKKS residues are < q_l)
 *   pt_diags        device, n_pt plaintexts of [L][N] uint64 NTT-domain
 *                   residues < 2^50, plaintext p starting at word p * pitch
 *                   (pitch = the plan's pt_pitch, L*N by default)
 *   ternary_groups  device, [n_member] int8 signs in {-1, 0, +1}, in the
 *                   member order of the layer description; must equal the
 *                   mem_sign the plan was created with (members that were 0
 *                   then are skipped; the others are read here)
 *   scales          device, [n_scale] uint64 integer reconstruction factors,
 *                   each < 2^20
 *   out_cts         device, [n_out][2][L][N] uint64, overwritten with
 *                   canonical residues in [0, q_l); must not overlap any input
 *   stream          HIP stream the work is queued on (0 = legacy default)
 * Asynchronous: returns once the kernel is queued; the buffers must stay
 * valid and unchanged until the stream reaches it.  Allocates nothing, and
 * issues kernel launches only (no memset or copy; a checking plan excepted),
 * so a call can be captured in a HIP graph.
 * Results are exact (bit-identical to evaluating every term on its own mod q_l).
 * Input ranges and signs above are preconditions, checked only by a checking
 * plan (FIONA_PLAN_CHECK_INPUTS).  Device pointers need 8-byte alignment
 * (every access is an 8-byte word).  Errors (nothing is launched):
 * FIONA_ERR_ARG (null pointer with a nonzero size), FIONA_ERR_ALIGN,
 * FIONA_ERR_ALIAS, FIONA_ERR_NODEVICE, FIONA_ERR_PRECONDITION (checking plans),
 * FIONA_ERR_HIP (launch, or a checking plan's copies).
 */
int fiona_hybrid_linear(const fiona_plan *plan, const uint64_t *in_cts, const uint64_t *pt_diags,
                        const int8_t *ternary_groups, const uint64_t *scales, uint64_t *out_cts,
                        hipStream_t stream);

/*
 * fiona_hybrid_linear_static: fiona_hybrid_linear for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, results and errors.
 * The per-call word blocks (the signed sums' member rows and the uses'
 * scales, written by the sign-packing kernel on every call) go to a
 * library-owned static device array of 4 MiB per device instead of the
 * plan's workspace; the array's address is looked up on the first call on a
 * device and kept until the process ends.  Allocates nothing (neither device
 * nor host memory).  Every call on one device shares its array and leaves its
 * blocks there; each call writes every block it reads before reading it, so
 * nothing needs clearing, but calls that overlap on one device (two streams,
 * or two host threads) race and must be serialized by the caller.
 * Errors, besides fiona_hybrid_linear's: FIONA_ERR_UNSUPPORTED if the plan's
 * word blocks exceed 4 MiB (more than 16384 common terms, resident sums and
 * uses); FIONA_ERR_ARG for a checking plan (FIONA_PLAN_CHECK_INPUTS), whose
 * check copies into host memory.
 */
int fiona_hybrid_linear_static(const fiona_plan *plan, const uint64_t *in_cts, const uint64_t *pt_diags,
                               const int8_t *ternary_groups, const uint64_t *scales, uint64_t *out_cts,
                               hipStream_t stream);

/*
 * Rescale epilogue: divide ciphertexts by the last modulus q_t = q_{L-1} of the
 * chain, with rounding, and drop that limb (CKKS rescaling, paper Sec. 2
 * "Levels and Bootstrapping").  Sec. 4.2 "Combining the Signed and Raw
 * Routes" rescales an output once, after its routes are summed: this is the
 * call that follows fiona_hybrid_linear.  Per coefficient, with C the integer
 * of the L residues: C' = round(C / q_t), kept as residues of the first L-1
 * moduli.
 *
 * NTT convention of every limb (input and output): a_hat_k = sum_n a_n
 * psi_l^((2k+1) n) mod q_l, k in natural order, psi_l a primitive 2N-th root
 * of unity mod q_l.
 *
 * fiona_rescaler_create: the NTT twiddle tables of every limb (device) and a
 * workspace for up to max_ct ciphertexts (2 * max_ct * N * 8 * (1 + k) bytes,
 * k = L - 1 limbs per launch, fewer when that would pass 8 GiB or 65535
 * vectors).
 *   psi     host [L] roots psi_l, or NULL for the default: psi_l =
 *           x^((q_l - 1) / 2N) for the smallest x >= 2 with psi_l^N = -1
 * Requires N a power of two in [2^8, 2^17], L >= 2, every q_l = 1 mod 2N and
 * max_ct <= 32767.
 * The rescaler keeps a reference to ctx (which must outlive it).  Errors:
 * FIONA_ERR_ARG, FIONA_ERR_UNSUPPORTED (N, L, a modulus or a root),
 * FIONA_ERR_NOMEM, FIONA_ERR_HIP.
 */
typedef struct fiona_rescaler fiona_rescaler;
int fiona_rescaler_create(const fiona_ctx *ctx, const uint64_t *psi, uint32_t max_ct, fiona_rescaler **out);
void fiona_rescaler_destroy(fiona_rescaler *rescaler);

/*
 * fiona_rescale: out = in / q_t with rounding, per ciphertext and polynomial.
 *   in_cts   device, [n_ct][2][L][N] uint64 canonical residues (NTT domain)
 *   out_cts  device, [n_ct][2][L-1][N] uint64, overwritten with canonical
 *            residues; must not overlap in_cts
 *   n_ct     at most the max_ct of the rescaler
 * Asynchronous on stream; allocates nothing, and issues kernel launches only
 * (no memset or copy), so a call can be captured in a HIP graph.  The
 * rescaler's workspace is shared by its calls: one rescaler must not be used
 * by two streams at the same time.  Errors (nothing is launched):
 * FIONA_ERR_ARG, FIONA_ERR_ALIGN, FIONA_ERR_ALIAS, FIONA_ERR_HIP.
 */
int fiona_rescale(const fiona_rescaler *rescaler, const uint64_t *in_cts, uint32_t n_ct, uint64_t *out_cts,
                  hipStream_t stream);

/*
 * Hoisted baby-step rotations: the step that produces fiona_hybrid_linear's
 * input ciphertexts.  A layer's inputs A_i are the packed input rotated by
 * the packing layout's baby steps (paper Sec. 2 "Homomorphic Operations": Rot
 * cyclically shifts the slots; Sec. 4.2: the A_i are prepared according to
 * the packing layout).  Rot by r slots is the automorphism sigma_g:
 * a(X) -> a(X^g), g = 5^r mod 2N (slot j of a message is its value at
 * zeta^(5^j), zeta = exp(i pi / N)), on both polynomials, followed by a key
 * switch of the second polynomial from sigma_g(s) back to s.  Key switching
 * decomposes c1 by RNS limb (digit j = the coefficients of c1 mod q_j, as
 * integers in [0, q_j)), multiplies digit j by key polynomial pair j over the
 * data moduli and one special prime P, sums, and divides by P with rounding:
 *     Rot(c0, c1) = (sigma(c0) + v_0, v_1),
 *     v_p = round(sum_j sigma(D_j) ksk[j][p] / P)    (coefficient-wise).
 * The digits are formed once per call and shared by all its rotations
 * (hoisting); the automorphism acts on the integer digits.  NTT convention:
 * as for the rescaler, for every modulus including P.
 *
 * fiona_rotator_create: NTT tables of q_0 .. q_{L-1} and P, and a workspace
 * for up to max_rot rotations per call (max_rot <= 256; about
 * 8 N (2 L (L + 1) + 2 L + max_rot (4 L + 4)) bytes).
 *   special_prime  P with 2^20 < P < 2^50, P = 1 mod 2N, unequal to every q_l
 *   psi            host [L + 1] roots (the data moduli, then P) or NULL for
 *                  the defaults of fiona_rescaler_create
 * Requires N a power of two in [2^8, 2^17], L + 1 <= FIONA_MAX_L and
 * max_rot <= 256.  Keeps a reference to ctx.  Errors: FIONA_ERR_ARG, FIONA_ERR_UNSUPPORTED,
 * FIONA_ERR_NOMEM, FIONA_ERR_HIP.
 *
 * Keys.  A rotation's key holds, for digit j < L and polynomial p in {0, 1},
 * one polynomial over the L + 1 moduli, NTT domain: [L][2][L + 1][N] uint64
 * canonical residues, modulus index L being P (fiona_rotation_key_words
 * words).  In its natural order, sum_j D_j ksk[j][0] + (sum_j D_j ksk[j][1]) s
 * = P D sigma_g(s) + small for a key that switches sigma_g(s) to s.
 * fiona_hoisted_rotate reads keys in the library's layout: each row of N
 * words permuted by the rotation's slot map and stored transposed (N = N1 N2
 * as in the NTT passes), written by fiona_rotation_key_layout from a key in
 * natural order (once per key).
 *
 * fiona_rotation_key_layout: key_out = the library layout of key (both device,
 *   fiona_rotation_key_words words, not overlapping) for Galois element
 *   galois (odd, < 2N).  Asynchronous on stream; allocates nothing.
 *
 * fiona_hoisted_rotate: n_rot rotations of one ciphertext.
 *   ct       device, [2][L][N] canonical residues (NTT domain)
 *   galois   host, [n_rot] Galois elements (odd, < 2N; 5^r mod 2N rotates by r)
 *   keys     device, [n_rot] keys in the library layout, key r for galois[r];
 *            16-byte aligned (read 16 bytes per lane)
 *   out_cts  device, [n_rot][2][L][N], overwritten with canonical residues;
 *            must not overlap ct or keys
 *   n_rot    at most the rotator's max_rot
 * Asynchronous on stream; allocates nothing, and issues kernel launches only
 * (the Galois elements travel by value in the launch arguments), so a call
 * can be captured in a HIP graph.  The workspace is shared by the rotator's
 * calls: one rotator must not be used by two streams at the same
 * time.  Results are exact: bit-identical to the definition above computed
 * in integers.  Errors (nothing is launched): FIONA_ERR_ARG, FIONA_ERR_ALIGN,
 * FIONA_ERR_ALIAS, FIONA_ERR_HIP.
 */
typedef struct fiona_rotator fiona_rotator;
int fiona_rotator_create(const fiona_ctx *ctx, uint64_t special_prime, const uint64_t *psi, uint32_t max_rot,
                         fiona_rotator **out);
void fiona_rotator_destroy(fiona_rotator *rotator);
uint64_t fiona_rotation_key_words(const fiona_rotator *rotator);
int fiona_rotation_key_layout(const fiona_rotator *rotator, uint32_t galois, const uint64_t *key,
                              uint64_t *key_out, hipStream_t stream);
int fiona_hoisted_rotate(const fiona_rotator *rotator, const uint64_t *ct, uint32_t n_rot, const uint32_t *galois,
                         const uint64_t *keys, uint64_t *out_cts, hipStream_t stream);

/*
 * Measurement helper (not part of the weighted sum): the register-only rate
 * of the raw route's arithmetic, against which the hybrid kernel's
 * multiply-add rate is compared.
 *
 * fiona_mac_microbench: launches blocks workgroups of 256 threads; every
 *   thread multiplies chunks * 56 plaintext words held in registers into both
 *   polynomials' exact accumulators, as the hybrid kernel does for one raw
 *   term at one position (four 32x32->64 multiply-adds per polynomial, a
 *   carry step every 56 words), reads no memory, and writes one word to
 *   sink[thread] (device, blocks * 256 words, caller-owned; the values mean
 *   nothing).  Asynchronous on stream; allocates nothing.  Errors:
 *   FIONA_ERR_ARG (blocks or chunks 0, sink NULL), FIONA_ERR_HIP.
 * fiona_mac_microbench_words: the plaintext words one such launch multiplies
 *   (blocks * 256 * chunks * 56).
 */
int fiona_mac_microbench(uint32_t blocks, uint32_t chunks, uint64_t *sink, hipStream_t stream);
uint64_t fiona_mac_microbench_words(uint32_t blocks, uint32_t chunks);

/*
 * Measurement helpers (not part of the weighted sum): the HBM bandwidth of a
 * plain contiguous read, of a plain copy and of a plain write, the ceilings
 * the kernels' rates are set against.  Grid-stride loops over 16-byte words
 * on blocks workgroups of 256 threads, nontemporal accesses.
 * fiona_stream_read: reads words (even) uint64 words of src (device, 16-byte
 *   aligned) and writes one word per workgroup to sink (device, blocks words).
 * fiona_stream_copy: dst[i] = src[i] for words (even) words (device, 16-byte
 *   aligned, not overlapping).
 * fiona_stream_write: writes words (even) words of dst (device, 16-byte
 *   aligned) with a pattern of the slot index; reads nothing.
 * Asynchronous on stream; allocate nothing.  Errors: FIONA_ERR_ARG,
 * FIONA_ERR_ALIGN, FIONA_ERR_ALIAS (copy), FIONA_ERR_HIP.
 */
int fiona_stream_read(const uint64_t *src, uint64_t words, uint32_t blocks, uint64_t *sink, hipStream_t stream);
int fiona_stream_copy(const uint64_t *src, uint64_t *dst, uint64_t words, uint32_t blocks, hipStream_t stream);
int fiona_stream_write(uint64_t *dst, uint64_t words, uint32_t blocks, hipStream_t stream);

/*
 * Checking helper (no device needed): replays the memory accesses of one
 * rescale (op 0) or one hoisted-rotation call (op 1) on the host.  The
 * rescaler (capacity = max_ct) or rotator (capacity = max_rot) is laid out
 * at fake device addresses, the call's launches are recorded instead of
 * issued, and every global access of every workgroup and thread of every NTT
 * pass is recomputed with the kernels' own offset arithmetic; the other
 * kernels of a rotation call are checked by the byte ranges they touch.
 *   moduli      host, L moduli (op 0) or L data moduli then the special
 *               prime (op 1), each = 1 mod 2N
 *   n_call      ciphertexts (op 0) or rotations (op 1) of the call; the
 *               rotations use Galois elements 5^r, then 2N - 1 and 1
 *   out_shrink  the caller's output buffer is taken to be this many bytes
 *               short (0 for the real size; a positive value checks that
 *               the checker finds the overrun)
 *   msg         host, msg_len bytes: the first violation, or ""
 * Returns FIONA_OK if every access lies inside the buffer that holds its
 * descriptor's base, below 2^32 bytes from it, with every descriptor's end
 * pointer at that buffer's end; FIONA_ERR_BOUNDS otherwise; the errors of
 * fiona_rescaler_create / fiona_rotator_create for bad parameters.
 */
int fiona_check_ntt_offsets(uint32_t op, uint32_t N, uint32_t L, const uint64_t *moduli, uint32_t capacity,
                            uint32_t n_call, uint64_t out_shrink, char *msg, size_t msg_len);

/* Static string naming a status code. */
const char *fiona_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* FIONA_H */
