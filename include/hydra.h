/*
 * hydra.h -- C ABI of the Hydra-PPO hot path on MI355X (gfx950).
 *
 * The operations follow "Efficient RLHF: Reducing the Memory Usage of PPO"
 * (arXiv 2309.00754):
 *   - LoRA on every linear layer of the actor and critic (Sec. 2, Stage 3);
 *   - Dynamic LoRA: the reference / reward model is the same network with the
 *     LoRA parameters ignored, LO(.) (Sec. 3, "Dynamic LoRA");
 *   - Hydra-PPO: one frozen base and two adapter sets, actor and critic; the
 *     active set is the one whose (A, B) pair is passed (Sec. 3, "Stage 2");
 *   - pi^hydra's two heads: a causal-LM head and a scalar reward head on the
 *     same input (Sec. 3, opening paragraph);
 *   - reward and reference log-probabilities from the LoRA-off model
 *     (App. A, Alg. 1 and Alg. 2).
 *
 * Conventions shared by every entry point
 *   - All tensor arguments are DEVICE pointers (hipMalloc'd or equivalent),
 *     row-major and contiguous.  bf16 values are passed as uint16_t bit
 *     patterns.  Operands read with 16-byte vector loads (x, W, A, h, W_lm,
 *     the fp32 logits and the workspace) must be 16-byte aligned; fp32 and
 *     int32 arrays 4-byte aligned; B and w_rm 2-byte aligned.
 *   - A linear layer's frozen weight W is stored output-major [N x K] (the
 *     nn.Linear.weight layout), LoRA-down A is [r x K], LoRA-up B is [N x r]:
 *         y_off = x W^T                     (LoRA off)
 *         y_on  = x W^T + s (x A^T) B^T     (LoRA on)
 *     Products are bf16 x bf16 with fp32 accumulation; outputs are fp32.
 *   - Ownership: the caller owns every buffer.  The library allocates no
 *     device memory and keeps no mutable global state; calls on different
 *     streams are independent.
 *   - Asynchrony: each call validates its arguments on the host, enqueues its
 *     kernels on `stream` (a hipStream_t; NULL = the default stream) and
 *     returns.  Inputs must stay valid until the stream reaches that point.
 *   - Errors: argument errors are detected on the host before any HIP call and
 *     returned as a negative status with nothing enqueued.  A failed launch
 *     returns HYDRA_ERR_HIP.  Data errors found on the device (a token id
 *     outside [0, V)) produce NaN in that token's outputs and OR 1 into
 *     *err_flag when err_flag is non-NULL.  NaN / Inf inputs propagate.
 *   - Results are deterministic: no floating-point atomics; every reduction
 *     runs in a fixed order, and the LoRA-on and LoRA-off log-softmax use
 *     identical reduction trees, so KL is exactly 0 wherever the two logit
 *     rows are equal (e.g. r = 0, s = 0 or B = 0).
 */
#ifndef HYDRA_H_
#define HYDRA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HYDRA_OK = 0,
  HYDRA_ERR_NULL = -1,        /* a required pointer is NULL                         */
  HYDRA_ERR_SHAPE = -2,       /* a size is out of range or inconsistent             */
  HYDRA_ERR_ALIGN = -3,       /* a pointer is not aligned as required               */
  HYDRA_ERR_UNSUPPORTED = -4, /* a valid request the library does not handle        */
  HYDRA_ERR_WORKSPACE = -5,   /* the workspace is missing or too small              */
  HYDRA_ERR_HIP = -6          /* the HIP runtime reported an error at launch        */
} hydra_status;

/* Largest LoRA rank accepted. */
#define HYDRA_MAX_RANK 128

/*
 * hydra_lora_linear -- the LoRA-switchable linear layer.
 * Defined by: Sec. 2 Stage 3 (LoRA on all linears), Sec. 3 "Dynamic LoRA"
 * (LO(.) = LoRA off on the same W) and "Stage 2: Hydra-PPO" (the adapter set
 * in use is the (A, B) passed).
 *
 *   x     [M x K] bf16   input rows (tokens)
 *   W     [N x K] bf16   frozen base weight, read once for both outputs
 *   A     [r x K] bf16   LoRA down projection (may be NULL iff r == 0)
 *   B     [N x r] bf16   LoRA up projection   (may be NULL iff r == 0)
 *   s     fp32           LoRA scale
 *   y_off [M x N] fp32   out: x W^T                  (NULL: not written)
 *   y_on  [M x N] fp32   out: x W^T + s (x A^T) B^T  (NULL: not written)
 * At least one output must be non-NULL.  Requires 1 <= M <= 2^20, 1 <= N <= 2^21,
 * K >= 1, K % 8 == 0, K <= 2^21, 0 <= r <= HYDRA_MAX_RANK, and
 * ceil(M / 128) * ceil(N / 256) < 2^23 (the GEMM's tile grid fits one
 * dispatch; roughly M * N < 2^38).  With r == 0, y_on equals
 * y_off.  M <= 16 selects the bandwidth-bound (decode) kernels, larger M the
 * MFMA GEMM; both compute the same function.  At M > 16 with y_on and r > 64
 * the update needs the pre-pass workspace of hydra_lora_linear_ws: this call
 * then returns HYDRA_ERR_WORKSPACE and launches nothing.
 */
hydra_status hydra_lora_linear(const uint16_t* x, const uint16_t* W, const uint16_t* A, const uint16_t* B,
                               float s, int64_t M, int64_t N, int64_t K, int64_t r,
                               float* y_off, float* y_on, void* stream);

/*
 * hydra_lora_linear_workspace_bytes -- device workspace that hydra_lora_linear_ws
 * needs for M rows, N outputs and rank r (0 when none is needed: r == 0).
 * Writes *bytes.  HYDRA_ERR_NULL for a NULL `bytes`, HYDRA_ERR_SHAPE for M
 * outside [1, 2^20], N outside [1, 2^21] or r outside [0, HYDRA_MAX_RANK].
 */
hydra_status hydra_lora_linear_workspace_bytes(int64_t M, int64_t N, int64_t r, size_t* bytes);

/*
 * hydra_lora_linear_ws -- hydra_lora_linear with a caller-provided workspace,
 * which lets the MFMA GEMM (M > 16) take the LoRA update from a pre-pass:
 * s x A^T is computed once per row (instead of once per 256-column tile) as
 * bf16 hi and lo parts, and added with B as 2 RP more k values of the GEMM
 * (RP = r rounded up to 16, 32, 64 or 128) after y_off has been stored.
 * This is the path for the paper's rank 128 (App. B), and the faster one
 * above rank 16, where the in-tile product of hydra_lora_linear adds RP / 256
 * of the base GEMM's work; at rank 16 the pre-pass costs about what the GEMM
 * saves.  Defined by: the same passages as hydra_lora_linear.
 *
 *   workspace, workspace_bytes   device memory of at least
 *       hydra_lora_linear_workspace_bytes(M, N, r) bytes, 16-byte aligned,
 *       contents ignored and overwritten; NULL allowed when that size is 0 or
 *       when no GEMM update runs (M <= 16, no y_on, or r == 0).
 * Other arguments and rules as in hydra_lora_linear; HYDRA_ERR_WORKSPACE for a
 * workspace that is needed and too small, HYDRA_ERR_ALIGN for a misaligned one.
 * y_off has the bits of hydra_lora_linear's; y_on agrees with it to the
 * rounding of T (different summation order).
 */
hydra_status hydra_lora_linear_ws(const uint16_t* x, const uint16_t* W, const uint16_t* A, const uint16_t* B,
                                  float s, int64_t M, int64_t N, int64_t K, int64_t r, float* y_off, float* y_on,
                                  void* workspace, size_t workspace_bytes, void* stream);

/* Largest number of linears in one hydra_lora_linear_group call. */
#define HYDRA_MAX_GROUP 8

/*
 * hydra_lora_linear_group -- G independent LoRA-switchable linears that share
 * M, N, K and r, in one launch (for instance the q/k/v/o projections of one
 * decode step, App. A Alg. 2, generation step; each with its own adapter).
 * Defined by: the same passages as hydra_lora_linear.
 *
 *   G                     1 <= G <= HYDRA_MAX_GROUP
 *   x, W, A, B, y_off, y_on   HOST arrays of G device pointers with the meaning,
 *                         layout and alignment of hydra_lora_linear's arguments;
 *                         A, B, y_off, y_on may be NULL arrays (all members NULL)
 *                         or hold NULL entries
 *   s                     HOST array of G scales
 * Member i computes exactly what hydra_lora_linear(x[i], W[i], A[i], B[i], s[i],
 * M, N, K, r, y_off[i], y_on[i]) computes.  Each member needs at least one
 * output.  M <= 16 runs one launch for the whole group; larger M runs the GEMM
 * once per member.  Errors as in hydra_lora_linear; HYDRA_ERR_SHAPE for G out
 * of range.
 */
hydra_status hydra_lora_linear_group(int64_t G, const uint16_t* const* x, const uint16_t* const* W,
                                     const uint16_t* const* A, const uint16_t* const* B, const float* s,
                                     int64_t M, int64_t N, int64_t K, int64_t r,
                                     float* const* y_off, float* const* y_on, void* stream);

/*
 * hydra_lora_linear_group_workspace_bytes -- device workspace that
 * hydra_lora_linear_group_ws needs for G linears of M rows, N outputs and
 * rank r (writes *bytes).  HYDRA_ERR_NULL for a NULL `bytes`, HYDRA_ERR_SHAPE
 * for G, M, N or r outside the limits of hydra_lora_linear_group.
 */
hydra_status hydra_lora_linear_group_workspace_bytes(int64_t G, int64_t M, int64_t N, int64_t r, size_t* bytes);

/* Control area at the start of a hydra_lora_linear_group_ws workspace, its caller-owned wait-bound word, the size
 * of the region of published T values that follows it, and the size of the region of published LoRA-off outputs
 * after that. */
#define HYDRA_GROUP_WS_CONTROL_BYTES 4352
#define HYDRA_GROUP_WS_BOUND_WORD 8
#define HYDRA_GROUP_WS_T_BYTES 65536
#define HYDRA_GROUP_WS_Y_BYTES 2097152

/*
 * hydra_lora_linear_group_ws -- hydra_lora_linear_group with a caller
 * workspace, which lets a decode step (M <= 8 rows, App. A Alg. 1 / Alg. 2,
 * generation step) run as a single launch: the first workgroups form
 * T = x A^T of every member once and publish it in the workspace; up to
 * padded rank 64 (when G x N x M, with M rounded up to 1, 2, 4 or 8, is at
 * most HYDRA_GROUP_WS_Y_BYTES / 8) the workgroups that stream the rows of W
 * publish their LoRA-off outputs there too, and workgroups at the end of the
 * launch add s T B^T to them to form y_on; otherwise the workgroups that stream W add
 * s T B^T to their own rows of y_on (no second launch, no T recomputed per
 * column block).  Defined by: the same passages as hydra_lora_linear.
 *
 *   G, x, W, A, B, s, M, N, K, r, y_off, y_on   as in hydra_lora_linear_group
 *   workspace, workspace_bytes   device, 16-byte aligned, at least
 *                         hydra_lora_linear_group_workspace_bytes(G, M, N, r)
 *                         bytes.  Fill the whole buffer with zeros once after
 *                         allocating it; after that the library keeps its
 *                         state there (HYDRA_GROUP_WS_CONTROL_BYTES of control
 *                         words holding a call generation, then
 *                         HYDRA_GROUP_WS_T_BYTES of published T values and
 *                         HYDRA_GROUP_WS_Y_BYTES of published LoRA-off outputs,
 *                         each tagged with it), so the buffer is reused as it
 *                         is and serves calls of any shape.  To reset it, zero all of
 *                         it (the control words alone are not enough), and
 *                         zero it again before its next use here after lending
 *                         it to another entry point.  One workspace serves one
 *                         stream at a time: calls that overlap in time must
 *                         not share it.  The 32-bit word
 *                         HYDRA_GROUP_WS_BOUND_WORD of the control area is the
 *                         caller's: 0 selects the default bounds of the
 *                         launch's waits (for T and for a published LoRA-off
 *                         output, about 10 ms each; for every workgroup to
 *                         have read the generation, about 1 s); another value
 *                         bounds each to that many polls.  A workgroup that
 *                         gives up waiting for T or for an output forms it
 *                         itself, with the same bits; if the last wait runs
 *                         out, every later call forms them where they are used
 *                         (same bits, slower) until the workspace is zeroed.
 * By rows: M <= 8 one launch; 8 < M <= 16 as hydra_lora_linear_group, but at
 * rank above 64 the two row halves each take the single launch; M > 16 as
 * hydra_lora_linear_group, and at rank above 64 each member runs the pre-pass
 * GEMM of hydra_lora_linear_ws over a pre-pass workspace of its own (one per
 * member, after the regions above); when every member's B has rows of exactly
 * the padded rank and is 16-byte aligned, the members' pre-passes share one
 * pair of launches before the GEMMs (rank 128 is accepted at every M).  Errors as in hydra_lora_linear_group, plus
 * HYDRA_ERR_NULL for a NULL workspace, HYDRA_ERR_WORKSPACE when it is too
 * small, HYDRA_ERR_ALIGN when it is not 16-byte aligned.  Results: the
 * oracle's tolerances; the bits may differ from hydra_lora_linear_group's in
 * y_on (another summation order of the LoRA update); repeated calls give the
 * same bits.
 */
hydra_status hydra_lora_linear_group_ws(int64_t G, const uint16_t* const* x, const uint16_t* const* W,
                                        const uint16_t* const* A, const uint16_t* const* B, const float* s,
                                        int64_t M, int64_t N, int64_t K, int64_t r,
                                        float* const* y_off, float* const* y_on,
                                        void* workspace, size_t workspace_bytes, void* stream);

/* Largest number of LoRA-on inputs in one hydra_lora_linear_multi call. */
#define HYDRA_MAX_ADAPTERS 4

/*
 * hydra_lora_linear_multi -- one frozen W serving a LoRA-off input and up to
 * HYDRA_MAX_ADAPTERS LoRA-on inputs, each with its own adapter.
 * Defined by: App. A, Alg. 2 (in each PPO iteration the same base weights run
 * the actor pass with the actor adapter, the critic pass with the critic
 * adapter, and the reference / reward passes with LoRA turned off, over the
 * same sequences), Sec. 3 "Dynamic LoRA" (LO(.) on the same W).  In a
 * multi-layer model the passes' activations differ after the first layer, so
 * every pass brings its own input.
 *
 *   x_off  [M x K] bf16 or NULL     input of the LoRA-off pass
 *   W      [N x K] bf16             frozen base weight
 *   n_on   0 <= n_on <= HYDRA_MAX_ADAPTERS
 *   x_on, A, B, y_on   HOST arrays of n_on device pointers: x_on[a] [M x K] bf16,
 *                      A[a] [r x K] bf16, B[a] [N x r] bf16, y_on[a] [M x N] fp32
 *                      (A and B may be NULL arrays iff r == 0)
 *   s      HOST array of n_on scales (NULL iff n_on == 0)
 *   y_off  [M x N] fp32  out: x_off W^T (NULL iff x_off is NULL)
 *   y_on[a]              out: x_on[a] W^T + s[a] (x_on[a] A[a]^T) B[a]^T
 * Shape, rank and alignment rules as in hydra_lora_linear; the outputs must be
 * distinct buffers (HYDRA_ERR_SHAPE otherwise) and at least one input given.
 * At M <= 8 the inputs' rows are stacked, at most 8 rows per pass, and each
 * pass reads W from HBM once for all its rows (M = 4 with the off input and
 * one adapter: one read of W instead of two); larger M runs one GEMM per input.
 * Every output has the bits of the corresponding hydra_lora_linear call.
 * Above M = 16 with adapters, a padded rank above 64 (r > 64) returns
 * HYDRA_ERR_WORKSPACE before anything is launched (hydra_lora_linear_multi_ws
 * serves that rank).
 */
hydra_status hydra_lora_linear_multi(const uint16_t* x_off, const uint16_t* W, int64_t n_on,
                                     const uint16_t* const* x_on, const uint16_t* const* A,
                                     const uint16_t* const* B, const float* s, int64_t M, int64_t N, int64_t K,
                                     int64_t r, float* y_off, float* const* y_on, void* stream);

/*
 * hydra_lora_linear_multi_workspace_bytes -- device workspace that
 * hydra_lora_linear_multi_ws needs for M rows, N outputs and rank r (writes
 * *bytes): the workspace of hydra_lora_linear_ws, shared by the adapters in
 * turn.  HYDRA_ERR_NULL / HYDRA_ERR_SHAPE as hydra_lora_linear_workspace_bytes.
 */
hydra_status hydra_lora_linear_multi_workspace_bytes(int64_t M, int64_t N, int64_t r, size_t* bytes);

/*
 * hydra_lora_linear_multi_ws -- hydra_lora_linear_multi with a caller
 * workspace, so that the paper's rank 128 (App. B) runs at every M.  Defined
 * by: the same passages as hydra_lora_linear_multi.
 *
 *   arguments as hydra_lora_linear_multi, plus
 *   workspace, workspace_bytes   device, 16-byte aligned, at least
 *                         hydra_lora_linear_multi_workspace_bytes(M, N, r)
 *                         bytes; its contents need not be anything in
 *                         particular, and the call overwrites them.
 * Above M = 16 with adapters at a padded rank above 64, the LoRA-off input runs
 * as hydra_lora_linear without an adapter and each adapter's input as
 * hydra_lora_linear_ws (the pre-pass GEMM), in turn over the workspace: every
 * output has the bits of that call.  Otherwise the call is
 * hydra_lora_linear_multi (the workspace is not used).  Errors as in
 * hydra_lora_linear_multi, plus HYDRA_ERR_NULL for a NULL workspace,
 * HYDRA_ERR_WORKSPACE when it is too small for the rank-128 case,
 * HYDRA_ERR_ALIGN when it is not 16-byte aligned; all before any launch.
 */
hydra_status hydra_lora_linear_multi_ws(const uint16_t* x_off, const uint16_t* W, int64_t n_on,
                                        const uint16_t* const* x_on, const uint16_t* const* A,
                                        const uint16_t* const* B, const float* s, int64_t M, int64_t N, int64_t K,
                                        int64_t r, float* y_off, float* const* y_on, void* workspace,
                                        size_t workspace_bytes, void* stream);

/*
 * hydra_score_workspace_bytes -- device workspace that hydra_score needs for
 * M = n_seq * seq_len token rows and a vocabulary of V.  Writes *bytes.
 * Returns HYDRA_ERR_NULL for a NULL `bytes`, HYDRA_ERR_SHAPE for M outside
 * [1, 2^20] or V outside [1, 2^21].
 */
hydra_status hydra_score_workspace_bytes(int64_t M, int64_t V, size_t* bytes);

/*
 * hydra_score -- fused two-head PPO scoring pass.
 * Defined by: Sec. 3 (pi^hydra's CLM head and reward head on the same input),
 * App. A Alg. 1 / Alg. 2 (the LoRA-off scoring step that yields the reward
 * and the reference log-probabilities; the actor log-probability is the
 * LoRA-on pass), App. B
 * (the KL penalty weight beta is applied by the caller, not here).
 *
 *   h        [M x K] bf16   final hidden states, M = n_seq * seq_len, sequence-major
 *   W_lm     [V x K] bf16   CLM head weight (output-major)
 *   A, B     [r x K], [V x r] bf16   LoRA of the CLM head (NULL iff r == 0)
 *   s        fp32           LoRA scale
 *   tokens   [M] int32      sampled token scored at each row (the caller applies
 *                           the usual next-token shift)
 *   w_rm     [K] bf16       reward head weight (no bias); NULL: reward not computed
 *   lp_on    [M] fp32       out: log softmax(z_on)[token],  z_on  = h W^T + s (h A^T) B^T
 *   lp_off   [M] fp32       out: log softmax(z_off)[token], z_off = h W^T
 *   kl       [M] fp32       out: lp_on - lp_off (per-token sampled KL estimate)
 *   reward   [n_seq] fp32   out: <h[b*seq_len + seq_len - 1], w_rm> (NULL: skipped)
 *   lse_on, lse_off [M] fp32  out, optional: log-sum-exp of each logit row
 *   workspace, workspace_bytes  device scratch of at least
 *                           hydra_score_workspace_bytes(M, V) bytes, 16-byte aligned
 *   err_flag [1] int32      optional device flag; 1 is OR-ed in for an out-of-range token
 * The [M x V] logits are never written to memory.  Requires K % 8 == 0,
 * K <= 2^21, 0 <= r <= HYDRA_MAX_RANK, 1 <= M <= 2^20, 1 <= V <= 2^21 and
 * ceil(M / 256) * ceil(V / 256) < 2^24 (the GEMM's tile grid fits one dispatch).
 */
hydra_status hydra_score(const uint16_t* h, const uint16_t* W_lm, const uint16_t* A, const uint16_t* B, float s,
                         const int32_t* tokens, const uint16_t* w_rm,
                         int64_t n_seq, int64_t seq_len, int64_t K, int64_t V, int64_t r,
                         float* lp_on, float* lp_off, float* kl, float* reward, float* lse_on, float* lse_off,
                         void* workspace, size_t workspace_bytes, int32_t* err_flag, void* stream);

/*
 * hydra_score_two_input -- the scoring pass when the actor pass and the
 * LoRA-off pass have their own final hidden states, as in a multi-layer model
 * (their activations differ after the first layer).
 * Defined by: App. A Alg. 2 (the actor pass runs with the actor's adapter, the
 * reference / reward pass with LoRA off, over the same sequences), Sec. 3
 * "Dynamic LoRA" (the reward model is the LoRA-off network), Sec. 3 (the two
 * heads of pi^hydra).
 *
 *   h_act    [M x K] bf16   final hidden states of the actor pass
 *   h_off    [M x K] bf16   final hidden states of the LoRA-off pass
 *   lp_on    [M] fp32       out: log softmax(z_on)[token],  z_on  = h_act W^T + s (h_act A^T) B^T
 *   lp_off   [M] fp32       out: log softmax(z_off)[token], z_off = h_off W^T
 *   kl       [M] fp32       out: lp_on - lp_off
 *   reward   [n_seq] fp32   out: <h_off[b*seq_len + seq_len - 1], w_rm> (NULL: skipped)
 *   every other argument    as in hydra_score (the same workspace size:
 *                           hydra_score_workspace_bytes(M, V))
 * One launch covers both inputs: the LoRA-off tile and the actor tile of a row
 * block run next to each other, so each block of W_lm is read from HBM once
 * for both.  The [M x V] logits are never written.  Errors as in hydra_score
 * (h_act is checked like h), plus HYDRA_ERR_SHAPE when
 * 2 * ceil(M / 256) * ceil(V / 256) >= 2^24.  With h_act and h_off equal the
 * results have the bits of hydra_score.
 */
hydra_status hydra_score_two_input(const uint16_t* h_act, const uint16_t* h_off, const uint16_t* W_lm,
                                   const uint16_t* A, const uint16_t* B, float s, const int32_t* tokens,
                                   const uint16_t* w_rm, int64_t n_seq, int64_t seq_len, int64_t K, int64_t V,
                                   int64_t r, float* lp_on, float* lp_off, float* kl, float* reward, float* lse_on,
                                   float* lse_off, void* workspace, size_t workspace_bytes, int32_t* err_flag,
                                   void* stream);

/* Largest workspace that hydra_score_noalloc serves from its own device scratch (48 MiB). */
#define HYDRA_SCORE_NOALLOC_MAX_BYTES (48u << 20)

/*
 * hydra_score_noalloc -- hydra_score without a caller workspace, for callers
 * that cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  The call itself allocates
 * nothing (no hipMalloc, hipFree or allocating library routine): the
 * workspace lives in a file-scope device array of the library,
 * HYDRA_SCORE_NOALLOC_MAX_BYTES long, one copy on each GPU the library runs
 * on, held until the process ends.  Its device address is looked up once per
 * device (on the first call there) and kept.
 *
 * Arguments, outputs and errors as in hydra_score, less `workspace` and
 * `workspace_bytes`; the caller still passes every input and output.
 * Returns HYDRA_ERR_WORKSPACE (before any HIP call) when
 * hydra_score_workspace_bytes(n_seq * seq_len, V) exceeds
 * HYDRA_SCORE_NOALLOC_MAX_BYTES (for example M = 2048, V = 32000 needs 21.5 MB
 * and fits; M = 4096, V = 50272 needs 44.6 MB and fits), and HYDRA_ERR_HIP if
 * the scratch's address cannot be found.  Results have the bits of hydra_score.
 * Every call on one GPU shares that GPU's scratch: calls that overlap in time
 * on one GPU (two streams, two host threads) race and give undefined results;
 * serialise them.  The scratch keeps the last call's contents; no call needs
 * it cleared.
 */
hydra_status hydra_score_noalloc(const uint16_t* h, const uint16_t* W_lm, const uint16_t* A, const uint16_t* B,
                                 float s, const int32_t* tokens, const uint16_t* w_rm,
                                 int64_t n_seq, int64_t seq_len, int64_t K, int64_t V, int64_t r,
                                 float* lp_on, float* lp_off, float* kl, float* reward, float* lse_on,
                                 float* lse_off, int32_t* err_flag, void* stream);

/*
 * hydra_score_logits -- the scoring epilogue alone, from materialised logits.
 * Defined by: App. A Alg. 2 (reference log-probabilities), Sec. 2 Stage 3
 * (the PPO policy ratio uses the same sampled-token log-probabilities).
 *
 *   logits_on, logits_off [M x V] fp32   logits of the LoRA-on and LoRA-off passes
 *   tokens   [M] int32                   sampled token per row
 *   lp_on, lp_off, kl [M] fp32           out (as in hydra_score)
 *   lse_on, lse_off [M] fp32             out, optional (NULL: not written)
 *   err_flag [1] int32                   optional, as in hydra_score
 * Requires 1 <= M <= 2^20 and 1 <= V <= 2^21.
 */
hydra_status hydra_score_logits(const float* logits_on, const float* logits_off, const int32_t* tokens,
                                int64_t M, int64_t V, float* lp_on, float* lp_off, float* kl,
                                float* lse_on, float* lse_off, int32_t* err_flag, void* stream);

/*
 * hydra_value_head -- the critic's scalar head on every token row.
 * Defined by: Sec. 2 Stage 3 (V(x, y) of the critic, used by generalized
 * advantage estimation), App. A Alg. 2 (the critic-LoRA pass over the
 * generated sequences that yields the values; h is that pass's final hidden
 * state).  No bias.
 *
 *   h       [M x K] bf16   hidden states, row-major, 16-byte aligned
 *   w_v     [K] bf16       value head weight, 16-byte aligned
 *   values  [M] fp32       out: values[m] = sum_k h[m][k] * w_v[k] (fp32 accumulation)
 * Requires 1 <= M <= 2^20, 1 <= K <= 2^21, K % 8 == 0.  Buffers are the caller's.
 */
hydra_status hydra_value_head(const uint16_t* h, const uint16_t* w_v, int64_t M, int64_t K, float* values,
                              void* stream);

/*
 * hydra_ppo_advantages -- per-token PPO reward and generalized advantage
 * estimates for n_seq sequences of seq_len tokens (M = n_seq * seq_len,
 * sequence-major).
 * Defined by: Sec. 2 Stage 3 (GAE builds the advantage estimates from the
 * reward using V; V is trained on the returns), App. A Alg. 2 (the advantage
 * step that combines the reward and the reference log-probabilities), App. B
 * (KL beta = 0.02,
 * GAE gamma = 1.0, lambda = 0.95).
 *
 *   kl      [M] fp32       per-token KL estimate lp_on - lp_off (hydra_score)
 *   reward  [n_seq] fp32   sequence reward (hydra_score), credited to the last token
 *   values  [M] fp32       critic values (hydra_value_head)
 *   start                  first response position, 0 <= start < seq_len
 *   beta, gamma, lam       KL weight and GAE discount / lambda
 *   rewards [M] fp32       out, optional: r_t = -beta * kl_t (t >= start) + (t == T-1) * reward
 *   advantages [M] fp32    out: A_t = delta_t + gamma * lam * A_{t+1},
 *                          delta_t = r_t + gamma * V_{t+1} - V_t, V_T = A_T = 0
 *   returns [M] fp32       out: A_t + V_t
 * Positions before `start` get advantage and return 0 (and reward 0).  No
 * output may be one of the inputs or another output (HYDRA_ERR_SHAPE);
 * partial overlaps are not detected and are not allowed.  Requires
 * n_seq, seq_len >= 1 and M = n_seq * seq_len <= 2^20 (HYDRA_ERR_SHAPE
 * otherwise, as for the other entry points' rows); buffers 4-byte aligned.
 */
hydra_status hydra_ppo_advantages(const float* kl, const float* reward, const float* values, int64_t n_seq,
                                  int64_t seq_len, int64_t start, float beta, float gamma, float lam, float* rewards,
                                  float* advantages, float* returns, void* stream);

/*
 * hydra_ppo_loss -- the PPO update stage's losses for n_seq sequences of
 * seq_len tokens (M = n_seq * seq_len, sequence-major), with their per-token
 * gradients.
 * Defined by: Sec. 2 Stage 3 (the clipped surrogate objective on the
 * probability ratio of the new and old policy; V trained with squared-error
 * loss on the returns).
 *
 *   lp_new, lp_old [M] fp32   sampled-token log-probabilities under the policy
 *                             being trained and under the one that sampled
 *   advantages, values, returns [M] fp32   A-hat (hydra_ppo_advantages), the
 *                             critic's current values, the returns
 *   start                     first response position, 0 <= start < seq_len
 *   eps                       clip range, 0 <= eps < 1 (the paper leaves it open)
 *   losses [3] fp32           out: policy loss -(1/n) sum min(rho A, clip(rho, 1-eps, 1+eps) A),
 *                             rho = exp(lp_new - lp_old); value loss (1/n) sum (V - R)^2 / 2;
 *                             the fraction of tokens where the clipped term is the smaller;
 *                             n = n_seq * (seq_len - start), the response tokens
 *   d_lp [M] fp32             out, optional: d policy loss / d lp_new (-rho A / n where the
 *                             unclipped term is the minimum, else 0; 0 before start)
 *   d_v [M] fp32              out, optional: d value loss / d V ((V - R) / n; 0 before start)
 * One workgroup sums in a fixed order (deterministic).  No output may be an
 * input or another output (HYDRA_ERR_SHAPE); buffers 4-byte aligned.
 * Requires n_seq, seq_len >= 1 and M = n_seq * seq_len <= 2^20.
 */
hydra_status hydra_ppo_loss(const float* lp_new, const float* lp_old, const float* advantages, const float* values,
                            const float* returns, int64_t n_seq, int64_t seq_len, int64_t start, float eps,
                            float* losses, float* d_lp, float* d_v, void* stream);

/*
 * hydra_transpose_bf16 -- dst = src^T for a bf16 matrix: src [R x C]
 * row-major, dst [C x R] row-major (dst[c * R + q] = src[q * C + c]).  The
 * update stage's backward reads the frozen base weight as W^T [K x N]; the
 * caller makes that copy once with this call (W does not change during
 * training) and keeps it beside W.
 *   src, dst   device, 2-byte aligned, not overlapping (HYDRA_ERR_SHAPE if equal)
 *   R, C       1 ... 2^21, ceil(R / 64) * ceil(C / 64) < 2^24
 * Bit-exact (a copy).
 */
hydra_status hydra_transpose_bf16(const uint16_t* src, int64_t R, int64_t C, uint16_t* dst, void* stream);

/*
 * hydra_lora_linear_backward_workspace_bytes -- device workspace that
 * hydra_lora_linear_backward needs for M rows, N outputs, K inputs and rank r
 * (0 for r == 0).  HYDRA_ERR_NULL for a NULL `bytes`, HYDRA_ERR_SHAPE for
 * sizes outside the limits of hydra_lora_linear_backward.
 */
hydra_status hydra_lora_linear_backward_workspace_bytes(int64_t M, int64_t N, int64_t K, int64_t r, size_t* bytes);

/*
 * hydra_lora_linear_backward -- gradients of the LoRA-on output
 * y = x W^T + s (x A^T) B^T with the base weight W frozen (the update stage
 * trains only the adapter: Sec. 3 and App. A, Alg. 2; LoRA as in Sec. 2):
 *   dx = dy W + s (dy B) A,   dA = s (dy B)^T x,   dB = s dy^T (x A^T).
 *
 *   x [M x K] bf16           the layer's input (device, 16-byte aligned)
 *   Wt [K x N] bf16          W transposed (hydra_transpose_bf16 of W [N x K]);
 *                            16-byte aligned; only read when dx is wanted
 *   A [r x K], B [N x r] bf16   the adapter (A 16-byte aligned, B 2-byte)
 *   s                        LoRA scale
 *   dy [M x N] bf16          gradient of the loss with respect to y (16-byte aligned)
 *   1 <= M <= 2^20; N, K >= 1, multiples of 8, at most 2^21;
 *   ceil(M / 128) * ceil(K / 256) < 2^23; 0 <= r <= HYDRA_MAX_RANK
 *   dx [M x K] fp32          out, optional
 *   dA [r x K] fp32          out, optional (ignored for r == 0)
 *   dB [N x r] fp32          out, optional (ignored for r == 0)
 *   workspace, workspace_bytes   device memory of at least
 *       hydra_lora_linear_backward_workspace_bytes(M, N, K, r) bytes, 16-byte
 *       aligned, contents ignored and overwritten (NULL allowed for r == 0)
 * dx comes from the MFMA GEMM of hydra_lora_linear_ws run on (dy, W^T) with
 * s (dy B) as its pre-pass; dA and dB are fp32 sums of outer products over
 * the M rows.  Every sum has a fixed order: repeated calls give the same bits.
 * At least one output is required (HYDRA_ERR_NULL); outputs 4-byte aligned
 * and distinct (HYDRA_ERR_SHAPE); HYDRA_ERR_WORKSPACE for a workspace that is
 * too small.  Calls that share a workspace on different streams race.
 */
hydra_status hydra_lora_linear_backward(const uint16_t* x, const uint16_t* Wt, const uint16_t* A, const uint16_t* B,
                                        float s, const uint16_t* dy, int64_t M, int64_t N, int64_t K, int64_t r,
                                        float* dx, float* dA, float* dB, void* workspace, size_t workspace_bytes,
                                        void* stream);

/* A static, human-readable name for a status code. */
const char* hydra_status_string(hydra_status status);

/* ABI version of this header (incremented on any incompatible change). */
int hydra_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* HYDRA_H_ */
