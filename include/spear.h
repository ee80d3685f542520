/*
 * spear.h -- C ABI of the MI355X (gfx950) W4+EC linear layer.
 *
 * The layer is the serving hot path of SPEAR (arXiv 2606.11244): a 4-bit
 * weight-only linear layer with the input-adaptive Error Compensator (EC)
 * folded in (section 3.1, Eq. 3):
 *
 *     Y = X . What^T + alpha * ( gate(X) (.) (X . A^T) ) . B^T
 *
 * with What[n][k] = (q[n][k] - z[n][k/G]) * s[n][k/G], the asymmetric
 * round-to-nearest 4-bit backbone of sections 2.1 and 5.1 (per output
 * channel, or per group of G input channels). The phase-aware dispatch of
 * section 4.1 chooses between a single fused kernel (decode, small M) and a
 * semi-fused EC pre-kernel + 4-bit GEMM whose epilogue adds the EC (prefill,
 * large M); spear_dispatch_plan exposes that choice.
 *
 * Conventions shared by every entry point:
 *   - Device pointers unless stated otherwise. Every device pointer must be
 *     16-byte aligned (SPEAR_E_ALIGN otherwise).
 *   - Row-major layouts, sizes in elements:
 *       x        [M][K]    activations, act dtype
 *       y        [M][N]    output, act dtype (overwritten, not accumulated)
 *       qweight  [N][K/8]  uint32; word j of row n holds code q[n][8j+i]
 *                          (0..15) in bits 4i..4i+3, lowest nibble first
 *                          (3-bit codes: [N][3K/32], see spear_w4_t)
 *       scales   [N][K/G]  IEEE fp16 bit patterns (both act dtypes)
 *       zeros    [N][K/G]  uint8, values 0..15
 *       A        [r][K]    act dtype      B  [N][r]  act dtype
 *       w_g      [K]       act dtype (sigmoid-linear gate)
 *       W1 [h][r], b1 [h], W2 [r][h], b2 [r]  act dtype (tanh-MLP gate)
 *   - Ownership: the caller owns every buffer; the library never allocates
 *     or frees device memory on these calls.
 *   - Errors: arguments are validated on the host before any launch; a
 *     validation failure returns a negative status and launches nothing. A
 *     failed launch returns SPEAR_E_HIP. Nothing is printed.
 *   - Asynchrony: every call is ordered on `hip_stream` (a hipStream_t; NULL
 *     means the default stream) and returns without synchronising.
 *   - Workspace: calls that need scratch take a caller-owned device buffer
 *     of at least spear_dispatch_plan()'s workspace_bytes. It must be
 *     zero-filled once before its first use. Its first 128 KiB hold counters:
 *     the split-K and EC-slice counters return to zero at the end of every
 *     call, and the fused path's launch-generation and ready counters advance
 *     by a fixed step per launch (their wrap-around is harmless). The next
 *     1 MiB holds the fused path's generation-tagged words and is written by
 *     no other kind of call; every call's other scratch data follows it. So
 *     the same workspace serves any later call (of any shape it is large
 *     enough for) and replays of a captured graph. Two calls that overlap in
 *     time must not share one workspace.
 */
#ifndef SPEAR_H
#define SPEAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t spear_status_t;

enum {
  SPEAR_OK = 0,
  SPEAR_E_NULL = -1,        /* a required pointer is NULL                   */
  SPEAR_E_SHAPE = -2,       /* M, N, K, G, r or h outside the supported set */
  SPEAR_E_DTYPE = -3,       /* unknown activation dtype, EC factor format or
                               weight code width                              */
  SPEAR_E_ALIGN = -4,       /* a device pointer is not 16-byte aligned      */
  SPEAR_E_WORKSPACE = -5,   /* workspace missing or smaller than required   */
  SPEAR_E_UNSUPPORTED = -6, /* gate kind or forced path not available       */
  SPEAR_E_HIP = -7,         /* a HIP launch or query failed                 */
  SPEAR_E_ALIAS = -8        /* the output overlaps an input                 */
};

/* Activation dtype: x, y, A, B and the gate parameters. */
enum { SPEAR_F16 = 0, SPEAR_BF16 = 1 };

/* Gate of the EC (section 3.1, Eq. 3). */
enum {
  SPEAR_GATE_ONE = 0,            /* gamma == 1: the static compensator of Eq. 2
                                    with W_comp = alpha B A                    */
  SPEAR_GATE_SIGMOID_LINEAR = 1, /* scalar per token g = sigmoid(w_g.x + b_g)  */
  SPEAR_GATE_TANH_MLP = 2        /* gamma = 1 + tanh(W2 ReLU(W1 A x + b1) + b2),
                                    the paper's rank-space gate (Eq. 3)        */
};

/* Execution path (section 4.1). AUTO lets spear_dispatch_plan choose by M. */
enum {
  SPEAR_PATH_AUTO = 0,
  SPEAR_PATH_FUSED_GEMV = 1,     /* one kernel: split-K 4-bit GEMV; the same grid
                                    computes A x and the gate, and the epilogue
                                    adds B (g (.) A x). Decode: up to 64
                                    tokens; AUTO's choice up to 32 where the
                                    local variant does not apply              */
  SPEAR_PATH_FUSED_MFMA = 2,     /* one kernel: the 4-bit MFMA GEMM also projects
                                    its activation tiles on A and w_g (split
                                    over K with the product when the tile grid
                                    is small), and its epilogue applies the
                                    gate and adds B (g (.) A x); rank <= 16,
                                    every gate (else SPEAR_E_UNSUPPORTED).
                                    AUTO picks it for
                                    M > 32 while the grid has at most 256
                                    128 x 128 tiles and the GEMM would not
                                    take 256-token tiles                       */
  SPEAR_PATH_UNFUSED_CHAIN = 3,  /* naive split: 4-bit GEMM, then separate
                                    projection, gate and reprojection+accumulate
                                    kernels (the baseline of section 4.1)      */
  SPEAR_PATH_UNFUSED_2K = 4,     /* semi-fused: EC pre-kernel (A x, gate) then
                                    the 4-bit GEMM/GEMV whose epilogue adds
                                    B (g (.) A x). AUTO's choice for M > 32
                                    otherwise                                  */
  SPEAR_PATH_OVERLAP_2K = 6,     /* semi-fused with the EC on a second stream
                                    (section 4.1's prefill design): the EC
                                    pre-kernel runs on a library-owned side
                                    stream concurrently with the 4-bit
                                    GEMM/GEMV on hip_stream; the side stream
                                    joins hip_stream before a final kernel adds
                                    B (g (.) A x) to Y. Three launches. The
                                    first call on a device creates the side
                                    stream and two events (so make it outside
                                    stream capture); calls from several host
                                    threads are serialised while they enqueue.
                                    AUTO does not pick it (measured slower)   */
  SPEAR_PATH_FUSED_LOCAL = 5     /* one kernel: split-K 4-bit GEMV whose waves
                                    also project x on [A; w_g] over their own K
                                    chunks (no EC workgroups, no wait on other
                                    workgroups beyond the split-K reduction);
                                    rank <= 16, every gate, M <= 32. AUTO
                                    picks it where it
                                    applies, otherwise SPEAR_PATH_FUSED_GEMV   */
};

typedef struct {
  int64_t M;            /* tokens, >= 0 (0 is a no-op)                        */
  int64_t N;            /* output features, >= 0 (0 is a no-op)               */
  int64_t K;            /* input features, a positive multiple of 128         */
  int32_t group_size;   /* G: 0 or K = per output channel; otherwise a
                           multiple of 128 that divides K                     */
  int32_t act_dtype;    /* SPEAR_F16 or SPEAR_BF16                            */
  int32_t rank;         /* r, 0..256 (0: the EC is absent)                    */
  int32_t gate_kind;    /* SPEAR_GATE_*                                       */
  int32_t gate_hidden;  /* h of the tanh-MLP gate, 0 = 4r; at most 1024       */
  int32_t force_path;   /* SPEAR_PATH_*; AUTO = choose by M                   */
  int32_t weight_bits;  /* code width of qweight: 0 or 4 (the default), or 3
                           (the 3-bit backbone of Appendix D.1 and D.3; zeros
                           then 0..7; layout at spear_w4_t); other values:
                           SPEAR_E_DTYPE                                      */
} spear_problem_t;

/* The quantised weight. 4-bit codes: qweight [N][K/8], word j of row n
 * holding q[n][8j+i] in bits 4i..4i+3. 3-bit codes (weight_bits = 3):
 * qweight [N][3K/32], the codes c_t = q[n][32j+t] (t = 0..31) of block j in
 * words 3j, 3j+1, 3j+2 of row n: word 3j holds the low two bits of c_{2i} in
 * bits 2i..2i+1 and of c_{2i+1} in bits 16+2i..17+2i (i = 0..7), word 3j+1
 * the same for c_{16+2i} and c_{17+2i}, word 3j+2 the high bit of c_{2i} in
 * bit i and of c_{2i+1} in bit 16+i (i = 0..15). */
typedef struct {
  const uint32_t* qweight; /* [N][K/8] (4-bit) or [N][3K/32] (3-bit) codes    */
  const uint16_t* scales;  /* [N][K/G] fp16 bits                              */
  const uint8_t* zeros;    /* [N][K/G] 0..15 (4-bit) or 0..7 (3-bit)          */
} spear_w4_t;

/* Storage of the EC factors A and B (section 5.1 and Appendix B.2: the
 * deployed compensators keep A and B in INT8, per output channel and
 * symmetric, and the gate in fp16). */
enum {
  SPEAR_AB_ACT = 0,  /* A, B in the activation dtype                          */
  SPEAR_AB_INT8 = 1  /* A, B int8 codes q in [-127, 127]: A[i][k] =
                        a_scale[i] * qA[i][k] (a_scale one fp32 per rank
                        channel), B[n][j] = b_scale[n] * qB[n][j] (one fp32
                        per output feature). Where a code feeds an MFMA it is
                        dequantised to the activation dtype, one rounding of
                        the fp32 product; where the kernel sums in fp32 (the
                        fused decode epilogue, the naive chain) the codes and
                        scale are used exactly                              */
};

typedef struct {
  const void* A;     /* [r][K] act dtype, or int8 (SPEAR_AB_INT8)             */
  const void* B;     /* [N][r] act dtype, or int8 (SPEAR_AB_INT8)             */
  float alpha;       /* EC scale (section 3.1); 1.0 when folded into B        */
  const void* w_g;   /* [K] act dtype      (SIGMOID_LINEAR only)              */
  float b_g;         /*                    (SIGMOID_LINEAR only)              */
  const void* W1;    /* [h][r] act dtype   (TANH_MLP only)                    */
  const void* b1;    /* [h]                                                   */
  const void* W2;    /* [r][h]                                                */
  const void* b2;    /* [r]                                                   */
  int32_t ab_format;       /* SPEAR_AB_*; other values: SPEAR_E_DTYPE       */
  const float* a_scale;    /* [r] fp32 (SPEAR_AB_INT8 only; 16-byte aligned) */
  const float* b_scale;    /* [N] fp32 (SPEAR_AB_INT8 only; 16-byte aligned) */
} spear_ec_t;

typedef struct {
  int32_t path;          /* resolved SPEAR_PATH_* (never AUTO)                */
  int32_t split_k;       /* K-slices of the 4-bit product (GEMV paths)        */
  int32_t ec_splits;     /* K-slices of the EC projection A x                 */
  int32_t tile_m;        /* tokens per workgroup tile                         */
  int32_t tile_n;        /* output rows per workgroup tile                    */
  int32_t num_launches;  /* kernel launches one call makes                    */
  int32_t grid;          /* workgroups of the main kernel                     */
  int32_t reserved;
  size_t workspace_bytes;/* scratch the call needs (0: none)                  */
} spear_plan_t;

/* Choose the execution path and launch shape for a problem (section 4.1:
 * fused for decode, semi-fused for prefill, switched by the token count M).
 * Host-only, pure and thread-safe: reads *prob, writes *out, touches no
 * device. `with_ec` = 0 plans spear_w4_linear, 1 plans spear_w4ec_linear.
 * Returns SPEAR_OK, or the validation error the call itself would return. */
spear_status_t spear_dispatch_plan(const spear_problem_t* prob, int32_t with_ec,
                                   spear_plan_t* out);

/* Y = X . What^T: the 4-bit weight-only linear layer with no EC (the
 * backbone of sections 2.1 and 5.1). The rank, gate and EC fields of *prob
 * are ignored. */
spear_status_t spear_w4_linear(const spear_problem_t* prob, const void* x,
                               const spear_w4_t* w, void* y, void* workspace,
                               size_t workspace_bytes, void* hip_stream);

/* Y = X . What^T + alpha * (gate (.) (X . A^T)) . B^T (section 3.1, Eq. 3),
 * executed on the path spear_dispatch_plan picks (or prob->force_path).
 * rank == 0 computes exactly what spear_w4_linear computes. */
spear_status_t spear_w4ec_linear(const spear_problem_t* prob, const void* x,
                                 const spear_w4_t* w, const spear_ec_t* ec,
                                 void* y, void* workspace,
                                 size_t workspace_bytes, void* hip_stream);

/* ---- Calls that allocate nothing --------------------------------------------
 * For callers that cannot allocate device memory or pass a workspace (code
 * under stream capture, serving loops or harnesses that forbid allocation):
 * spear_w4ec_linear with the scratch taken from a static array inside the
 * library, SPEAR_SCRATCH_BYTES per GPU, held from the library's load until
 * the process ends (one copy per device, found on the first call on each
 * device). Same arguments, path, kernels and results as spear_w4ec_linear
 * (bit for bit); the call allocates nothing and issues no memset (the array's
 * counters start at zero when the library is loaded, and every call leaves
 * them ready for the next). Problems whose planned workspace_bytes exceed
 * SPEAR_SCRATCH_BYTES return SPEAR_E_WORKSPACE; SPEAR_E_HIP if the scratch
 * cannot be located on the current device. Every call on one GPU uses the
 * same array: calls that overlap in time on one GPU (other streams, other
 * host threads) race and must be serialised by the caller. */
#define SPEAR_SCRATCH_BYTES (16u << 20)

spear_status_t spear_w4ec_linear_noalloc(const spear_problem_t* prob, const void* x,
                                         const spear_w4_t* w, const spear_ec_t* ec, void* y,
                                         void* hip_stream);

/* Post-EC tail (section 4.2: after the compensated product, the residual
 * addition and the next layer's RMSNorm). */
typedef struct {
  const void* residual;  /* [M][N] act dtype, added to Y before Y's single
                            rounding (Y becomes the new hidden state); may
                            be Y itself (in place); NULL: no residual        */
  const void* norm_w;    /* [N] act dtype: the next layer's RMSNorm weight;
                            NULL: no norm                                    */
  float eps;             /* RMSNorm epsilon, finite and >= 0                 */
  void* y_norm;          /* [M][N] act dtype: Y[m][n] * w[n] /
                            sqrt(mean_n Y[m][n]^2 + eps) over the stored Y,
                            computed in fp32 and rounded once; required with
                            norm_w; overlaps nothing else                    */
} spear_tail_t;

/* spear_w4ec_linear (or, with ec == NULL, spear_w4_linear) followed by the
 * post-EC tail. The residual is added inside the layer's own final store on
 * every path (the naive chain: in its 4-bit kernel); the RMSNorm, which needs
 * each token's whole row of Y while the layer's workgroups each hold a
 * slice of it, runs as one more kernel (one workgroup per token) in the same
 * call. The workspace is the one spear_dispatch_plan gives for the call
 * (with_ec = ec != NULL). Errors as for the layer call, plus SPEAR_E_NULL for
 * a missing tail or y_norm, SPEAR_E_ALIGN for a misaligned tail pointer,
 * SPEAR_E_ALIAS for y_norm overlapping another buffer or a residual that
 * overlaps Y without being Y, SPEAR_E_SHAPE for a negative or non-finite
 * eps. */
spear_status_t spear_w4ec_linear_tail(const spear_problem_t* prob, const void* x,
                                      const spear_w4_t* w, const spear_ec_t* ec,
                                      const spear_tail_t* tail, void* y, void* workspace,
                                      size_t workspace_bytes, void* hip_stream);

/* ---- Grouped calls ---------------------------------------------------------
 * At decode a layer call is a few microseconds of latency around a few MB of
 * weights (section 4.1: launch overhead, not arithmetic, dominates the decode
 * path), and the modules of a transformer block that read the same hidden
 * state (q, k, v; gate, up) are independent calls. A group runs up to
 * SPEAR_GROUP_MAX such calls, and the members that take one single-launch
 * GEMV variant share one launch: the 4-bit product alone (ec NULL) or the
 * fused local path (M <= 32, an elementwise gate and rank <= 16, where the
 * planner takes that path), with the same act dtype, code width and token
 * tiles. Of several such sets the largest (at least two members) shares the
 * launch. Its members are re-planned to one row-tile count where their own
 * plans differ and the re-plan leaves every member's K-slices and per-wave
 * work unchanged (the largest such count); local-EC members whose blocks
 * together exceed one round on the GPU then take four row tiles each under
 * the same condition. The other members (other variants, token counts
 * beyond the GEMV, a tiling that cannot be shared) run first, one after
 * another in array order on the same stream, each on its own planned path.
 * Either way each member's Y is exactly (bit for bit) what its own
 * spear_w4ec_linear or spear_w4_linear call writes. */
#define SPEAR_GROUP_MAX 4

/* One member: a problem and its operands as in spear_w4ec_linear; ec NULL
 * runs the 4-bit product alone (spear_w4_linear). Host struct; the pointers
 * inside follow the single calls' conventions. */
typedef struct {
  const spear_problem_t* prob;
  const void* x;
  const spear_w4_t* w;
  const spear_ec_t* ec; /* or NULL */
  void* y;
} spear_layer_call_t;

/* Workspace bytes of a group. Every nonempty workspace layout starts with
 * the same counter block and tagged region (the first 1152 KiB); a group's
 * workspace is those followed by each member's data region (its plan's bytes
 * past them, rounded up to 256) in array order, so it is at least every
 * member's own size and, like a single call's, may be shared in stream order
 * with single calls and other groups. 0 when no member needs scratch.
 * Host-only. SPEAR_E_NULL for a NULL array, member problem or out pointer,
 * SPEAR_E_SHAPE for n outside [1, SPEAR_GROUP_MAX], and every code
 * spear_dispatch_plan returns for a member. */
spear_status_t spear_group_workspace(int32_t n, const spear_layer_call_t* calls, size_t* out_bytes);

/* Kernel launches a spear_w4ec_linear_group call with these members makes:
 * one for the members that share a launch, plus each other member's own
 * launch count (spear_plan_t.num_launches). Host-only. Errors as in
 * spear_group_workspace. */
spear_status_t spear_group_launches(int32_t n, const spear_layer_call_t* calls, int32_t* out_launches);

/* Runs the n members (see above) on hip_stream. Validation of every member
 * (the single calls' checks) happens before any launch; in addition each
 * member's Y may not overlap any buffer of another member (SPEAR_E_ALIAS);
 * members may share X. Members with M == 0 or N == 0 are skipped. The
 * workspace (at least spear_group_workspace's bytes, zero-filled once before
 * first use) follows the single calls' rules: calls that overlap in time
 * need separate workspaces. */
spear_status_t spear_w4ec_linear_group(int32_t n, const spear_layer_call_t* calls, void* workspace,
                                       size_t workspace_bytes, void* hip_stream);

/* Diagnostic of the dequantisation the kernels use: writes
 * w_out[n][k] = RNE_act((q[n][k] - z[n][k/G]) * s[n][k/G]) as a dense [N][K]
 * act-dtype matrix, the exact product rounded once to nearest even
 * (sections 2.1, 5.1). Only N, K, group_size and act_dtype of *prob are
 * read. */
spear_status_t spear_w4_dequant(const spear_problem_t* prob, const spear_w4_t* w,
                                void* w_out, void* hip_stream);

/* Workspace layout of a planned call, for tests of its invariants (host
 * only): the fused path's tagged words occupy [*tag_begin, *tag_end) (both 0
 * on every other path), a region at a fixed place past the counter block
 * that no other kind of call writes; the call's other data regions lie in
 * [*data_begin, *data_end) (both 0 when it has none), which starts past the
 * tagged region for every call. Returns spear_dispatch_plan's status;
 * SPEAR_E_NULL for a NULL pointer. */
spear_status_t spear_workspace_regions(const spear_problem_t* prob, int32_t with_ec,
                                       size_t* tag_begin, size_t* tag_end, size_t* data_begin,
                                       size_t* data_end);

/* Test hook for the fused path's bounded wait: the number of polls a
 * workgroup makes for the EC coordinates before computing them itself
 * (default 1 << 16; 0 forces every workgroup onto that self-computing
 * fallback). Process-wide; returns the previous value. */
int32_t spear_set_wait_polls(int32_t polls);

/* Tuning hook for the decode GEMV's launch shape, process-wide: 16-row
 * tiles per workgroup (1, 2 or 4 for up to 32 tokens; 1 or 2 above), K-slices
 * per row group, and waves per workgroup (1..8). 0 restores the planner's
 * choice for that field. A combination that is not compiled in makes the
 * planner and the calls return SPEAR_E_UNSUPPORTED. For measurement sweeps
 * only. */
void spear_set_gemv_shape(int32_t row_tiles, int32_t k_slices, int32_t waves);

/* Tuning hook for the decode GEMV's pipeline depth, process-wide: stages of
 * packed codes in flight per wave, 2 or 4 (4: one token tile, the 4-bit
 * product alone, the producer-fused and the semi-fused variants; else the
 * planner and the calls return SPEAR_E_UNSUPPORTED); 0 restores the
 * planner's choice. For measurement sweeps and tests only. */
void spear_set_gemv_stages(int32_t stages);

/* Tuning hook for the prefill GEMM's K-slices (1, 2, 4 or 8; each slice an
 * even number of 64-wide K steps, else the planner and the calls return
 * SPEAR_E_UNSUPPORTED), process-wide; 0 restores the planner's choice (more
 * slices only while the tile grid alone leaves CUs idle). For measurement
 * sweeps and tests only. */
void spear_set_gemm_slices(int32_t k_slices);

/* Tuning hook for the prefill GEMM's token tile, process-wide: 128 (four
 * waves, two workgroups per CU) or 256 (eight waves, one workgroup per CU;
 * not the fully fused path: SPEAR_E_UNSUPPORTED there); any other value
 * restores the planner's choice (256 while those tiles fill the 256 CUs,
 * each 4096 of K beyond the first counting as another round of tiles). For
 * measurement sweeps and tests only. */
void spear_set_gemm_tile(int32_t tokens);

/* Tuning override of the prefill GEMM's wave roles: 1 = every wave loads,
 * dequantises and multiplies (k_gemm); 2 = four loading and four
 * multiplying waves on 256 x 128 tiles, 3 = four loading and eight
 * multiplying waves on 256 x 256 tiles (k_gemm_ws: 256-token tiles, one
 * K-slice, the plain and semi-fused epilogues; planning a problem
 * that does not allow them then returns SPEAR_E_UNSUPPORTED); 0 restores the
 * planner's choice (3 where 256 x 256 tiles fill the 256 CUs, else 2, where
 * allowed). For measurement sweeps and tests only. */
void spear_set_gemm_roles(int32_t roles);

/* Static text for a status code. */
const char* spear_status_string(spear_status_t status);

/* Library version, e.g. "0.1.0". */
const char* spear_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SPEAR_H */
