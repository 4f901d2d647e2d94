/*
 * asymspec.h -- C ABI of the AsymSpec fused decision step for MI355X (gfx950).
 *
 * AsymSpec ("Context-Asymmetric Speculative Decoding for Agentic LLMs",
 * arXiv 2608.26004) runs three forwards per speculative step: the drafter on
 * the full context (logits a, drafts d_1..d_K), the same drafter on the
 * compressed context (logits b) and the verifier on the compressed context
 * (logits t), each at the K+1 speculated positions (Sec. 3.2; Alg. 1).  This
 * library is the step that consumes those logits:
 *
 *   delta_i    = a_i - b_i                                  (Sec. 3.2, Eq. 1)
 *   f_i        = t_i + beta * delta_i      fused logits     (Sec. 3.2, Eq. 2)
 *   D_i        = JSD(softmax(a_i) || softmax(b_i))          (Sec. 3.3, Eq. 3)
 *   gamma_eff  = gamma * exp(-D_i)          CDA gate        (Sec. 3.3, Eq. 3)
 *   accept d_i iff softmax(t_i)[d_i] > gamma_eff * softmax(b_i)[d_i]  (Eq. 4)
 *   first rejection at j: emit argmax f_j; all accepted: emit argmax t_K
 *                                                           (Alg. 1)
 *   (argmax f_K instead with the ASYMSPEC_FUSE_BONUS flag)
 *
 * The paper defines the step for greedy decoding (temperature 0).  For a
 * request with temperature tau > 0 the library uses the speculative-sampling
 * form of the same gate: fused target p~ = softmax(f/tau), proposal
 * q = softmax(a/tau); accept d_i iff u_i < min(1, p~(d_i) / (gamma_eff q(d_i)));
 * at the first rejection the emitted token is an inverse-CDF draw from the
 * residual max(0, p~ - q) with the caller uniform u_K; when all drafts pass it
 * is an inverse-CDF draw from softmax(t_K/tau) with u_K.  With a == b and
 * gamma = 1 this is exactly standard speculative sampling.
 *
 * Conventions
 *   - Every pointer argument of asymspec_fuse_verify is a DEVICE pointer owned
 *     by the caller.  The library allocates, frees and retains nothing on this
 *     path; outputs are overwritten.
 *   - Calls are asynchronous: work is enqueued on `stream` (a hipStream_t, or
 *     NULL for the default stream) and the call returns; outputs are valid
 *     once the stream has been synchronised.
 *   - Errors are returned as negative status codes; argument checks happen on
 *     the host before anything is enqueued.  No exception crosses the ABI.
 *   - Layout: contiguous row-major; logits are [B][K+1][V] with row stride V;
 *     any V >= 1.  Row K of a and b is read only with ASYMSPEC_FUSE_BONUS (the
 *     bonus token of Alg. 1 uses the verifier alone).
 *   - Masked tokens: -inf logits are allowed.  A token whose fused logit is
 *     not a number (a = b = -inf) counts as masked.  NaN inputs otherwise give
 *     unspecified outputs.  Every row that is read must hold a finite logit.
 */
#ifndef ASYMSPEC_H
#define ASYMSPEC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------- */
#define ASYMSPEC_OK            0
#define ASYMSPEC_E_ARG        -1  /* null pointer, size or parameter out of range */
#define ASYMSPEC_E_ALIGN      -2  /* a pointer is not aligned as documented         */
#define ASYMSPEC_E_WORKSPACE  -3  /* workspace smaller than asymspec_workspace_size */
#define ASYMSPEC_E_DEVICE     -4  /* no gfx950 device current, or launch failure     */

/* ---- logit storage types --------------------------------------------- */
#define ASYMSPEC_BF16 0           /* bfloat16 bit patterns, 2 bytes per logit */
#define ASYMSPEC_FP32 1           /* IEEE binary32, 4 bytes per logit         */

/* ---- acceptance gates -------------------------------------------------- */
#define ASYMSPEC_GATE_CDA    0    /* gamma_eff = gamma * exp(-JSD)   (Eq. 3)          */
#define ASYMSPEC_GATE_FIXED  1    /* gamma_eff = gamma, the fixed-gamma gate the paper
                                     compares against (App. B, "Models and
                                     hyperparameters") */
#define ASYMSPEC_GATE_KL     2    /* gamma_eff = gamma * exp(-KL(P || Q)), P and Q the
                                     drafter views' softmaxes: the KL instantiation of
                                     D in the JSD-vs-KL table (App. G); not bounded */
#define ASYMSPEC_GATE_LAMBDA 3    /* gamma_eff = gamma * exp(-lambda * Delta(d)),
                                     Delta = log softmax(a) - log softmax(b) at the
                                     draft token: the tuned-lambda gate (App. B) */

/* ---- sources of the context-gain signal delta (Eq. 1-2) ---------------- */
#define ASYMSPEC_DELTA_AB 0       /* delta = a - b (Eq. 1, the paper's method)        */
#define ASYMSPEC_DELTA_A  1       /* delta = a, raw-augmented (Sec. 6.2 ablation)     */
#define ASYMSPEC_DELTA_TB 2       /* delta = t - b, SCD-style (Sec. 6.2 ablation)     */

/* ---- flags ------------------------------------------------------------- */
#define ASYMSPEC_FUSE_BONUS 1u    /* the bonus token comes from the fused row
                                     f_K = t_K + beta delta_K (greedy argmax, or a
                                     draw from softmax(f_K/tau)) instead of t_K.
                                     Alg. 1 appends argmax t_{K+1}, but the drafter
                                     logits of position K+1 exist (Alg. 1 computes
                                     a and b over all K+1 positions); this reads
                                     rows K of a and b as well */

#define ASYMSPEC_EARLY_EXIT 2u    /* Alg. 1 stops at the first rejection: the first
                                     early_rows rows of a request are read and
                                     classified first, and the other rows are read
                                     only if none of those is surely rejected.
                                     accept_len, next_token and fused_logprobs[K]
                                     are unchanged; fused_logprobs[i] and gate_out[i]
                                     of rows not read (all after the first rejection)
                                     are NaN.  Not with fused_logprobs_full */

typedef struct asymspec_params {
  float beta;         /* fusion weight of Eq. 2; finite, >= 0 (paper default 1.0) */
  float gamma;        /* base threshold of Eq. 3-4; in (0, 1] (paper default 0.5)  */
  int32_t gate_mode;  /* ASYMSPEC_GATE_*                                           */
  uint32_t flags;     /* ASYMSPEC_FUSE_BONUS | ASYMSPEC_EARLY_EXIT; other bits 0     */
  int32_t delta_mode; /* ASYMSPEC_DELTA_* (ASYMSPEC_DELTA_AB for the paper)        */
  float lambda;       /* scale of ASYMSPEC_GATE_LAMBDA, finite (paper default 0.1);
                         ignored by the other gates                                */
  int32_t early_rows; /* with ASYMSPEC_EARLY_EXIT: rows read before the verdict, in
                         [0, 63] (0: 2); early_rows >= K + 1 reads every row        */
} asymspec_params;

/* Bytes of device workspace asymspec_fuse_verify needs for this shape
 * (0 for invalid arguments).  The workspace needs no initialisation and may be
 * reused across calls of any shape: every record the kernel exchanges between
 * workgroups is tagged with a per-call epoch.
 * Calls that may run at the same time need distinct workspaces.
 * The epoch is a launch argument chosen on the host at each call, so a call
 * must not be captured into a HIP graph and replayed: every replay would
 * reuse one epoch and could take the previous replay's records for its own. */
size_t asymspec_workspace_size(int B, int K, int V, int dtype);

/* Zero-fill a workspace on `stream` with a fill kernel (never required for
 * correctness; useful to scrub a buffer).  Returns ASYMSPEC_OK, ASYMSPEC_E_ARG
 * or ASYMSPEC_E_DEVICE. */
int asymspec_workspace_clear(void* workspace, size_t workspace_bytes, void* stream);

/*
 * One decision step (Alg. 1, the body of the while loop after the three
 * forwards) for B independent requests with K drafts each.
 *
 *   verifier_logits     t [B][K+1][V]  (dtype)          16-byte aligned
 *   drafter_full_logits a [B][K+1][V]  (dtype)          16-byte aligned; rows 0..K-1 read,
 *                                                       row K too with ASYMSPEC_FUSE_BONUS
 *   drafter_comp_logits b [B][K+1][V]  (dtype)          same as a
 *                       (a and b may be NULL when K = 0 without ASYMSPEC_FUSE_BONUS)
 *   draft_tokens        d [B][K] int32, each in [0, V)  (may be NULL when K = 0)
 *   draft_probs         q(d) [B][K] float, or NULL: the proposal probability of
 *                       each draft for sampling rows; NULL means softmax(a/tau)[d]
 *                       computed here.  Unused on greedy rows.
 *   uniforms            u [B][K+1] float in [0,1): u[b][i] (i < K) decides the
 *                       acceptance of draft i on sampling rows, u[b][K] drives the
 *                       emission draw.  Unused for greedy requests, but required.
 *   temperature         tau [B] float; tau <= 0 selects greedy decoding for
 *                       that request (the paper's setting), tau > 0 sampling.
 *   B >= 1, 0 <= K <= 63, V >= 1, B*(K+1)*V < 2^40, and V at most
 *                       4194297 (bf16) or 2097149 (fp32): a row spans at most
 *                       256 chunks of 32 KiB
 *   params              see asymspec_params (host pointer)
 *   accept_len          [B] int32 out: number of accepted drafts, in [0, K]; -1
 *                       marks a request whose decision did not complete
 *                       (asymspec_workspace_timeouts)
 *   next_token          [B] int32 out: the token emitted after them
 *   fused_logprobs      [B][K+1] float out: [i] (i < K) = log p~_i(d_i), the
 *                       fused log-probability of draft i (temperature 1 for
 *                       greedy requests, tau for sampling ones); [K] = the
 *                       log-probability of next_token under the distribution
 *                       that emitted it (the fused row at the first rejection,
 *                       or the bonus row: t_K, or f_K with ASYMSPEC_FUSE_BONUS)
 *   gate_out            [B][K][2] float out (D_i, gamma_eff_i), or NULL; D_i
 *                       is the JSD (CDA and fixed gates), the KL (KL gate) or
 *                       lambda * Delta_i(d_i) (lambda gate), and gamma_eff_i =
 *                       gamma (fixed gate) or gamma * exp(-D_i)
 *   fused_logprobs_full [B][K+1][V] float out, or NULL; 16-byte aligned.  Every
 *                       element's log-probability under its row's distribution:
 *                       rows i < K log softmax(f_i/tau), row K log softmax(t_K/tau)
 *                       (of f_K with ASYMSPEC_FUSE_BONUS), tau = 1 for greedy
 *                       requests; -inf where f is not a number.  Written by a
 *                       second kernel on `stream` that reads the logits again
 *                       (3 (K+1) V elements) and writes 4 (K+1) V bytes per request;
 *                       one workgroup per 32 KiB chunk of a row, so B (K+1) times
 *                       the chunks per row must stay below 2^31 (else E_ARG)
 *   workspace           device scratch of >= asymspec_workspace_size bytes,
 *                       256-byte aligned, contents opaque between calls
 *   stream              hipStream_t or NULL
 *
 * Integer and float arrays must be 4-byte aligned.  Returns ASYMSPEC_OK or a
 * negative status; on error nothing is enqueued.  A request whose outputs
 * could not be completed on the device (a wait between workgroups timed out,
 * counted in the workspace: asymspec_workspace_timeouts) has accept_len = -1.
 */
int asymspec_fuse_verify(const void* verifier_logits,
                         const void* drafter_full_logits,
                         const void* drafter_comp_logits,
                         int dtype,
                         const int32_t* draft_tokens,
                         const float* draft_probs,
                         const float* uniforms,
                         const float* temperature,
                         int B, int K, int V,
                         const asymspec_params* params,
                         int32_t* accept_len,
                         int32_t* next_token,
                         float* fused_logprobs,
                         float* gate_out,
                         float* fused_logprobs_full,
                         void* workspace, size_t workspace_bytes,
                         void* stream);

/*
 * The same step for a drafter and a verifier with different vocabularies
 * (Sec. 6.4 and App. D): delta is computed in the
 * drafter's vocabulary and carried to the verifier's through the
 * string-identical tokens the two share, and committed tokens are restricted
 * to that shared set.
 *
 *   verifier_logits     t [B][K+1][V] in the verifier's vocabulary, 16-byte aligned
 *   drafter_full_logits a [B][K+1][Vd] in the drafter's vocabulary, 4-byte aligned
 *   drafter_comp_logits b [B][K+1][Vd], 4-byte aligned
 *   vocab_map           [V] int32 device array: vocab_map[x] is the drafter id of
 *                       verifier token x, or -1 when x has no shared counterpart
 *                       (entries outside [0, Vd) count as -1); 4-byte aligned
 *   Vd                  drafter vocabulary size, B*(K+1)*Vd < 2^40
 *   workspace           >= asymspec_workspace_size_xvocab(B, K, V, Vd, dtype) bytes
 *   draft_tokens        verifier ids of the drafts
 *   everything else     as for asymspec_fuse_verify
 *
 * Reading: every distribution of the step is taken over the shared set, as
 * if each row were first carried into the verifier's vocabulary with the
 * tokens outside the set masked in all three views: f(x) = t(x) + beta delta
 * (vocab_map[x]), the log-softmaxes of Eq. 3-4 (so D and p_b), the sampling
 * target and proposal, the emission and the bonus token.  Drafter tokens
 * that no verifier token maps to are never read.  A draft outside the set has
 * no mass in any view and is rejected.  The drafter rows are gathered element
 * by element (a map is in general no permutation of contiguous runs); when
 * no two verifier tokens share a drafter id, rows with no argmax to find read
 * the drafter rows in their own order and gather t instead.
 */
/* Workspace bytes of asymspec_fuse_verify_xvocab (0 for invalid arguments). */
size_t asymspec_workspace_size_xvocab(int B, int K, int V, int Vd, int dtype);

int asymspec_fuse_verify_xvocab(const void* verifier_logits,
                                const void* drafter_full_logits,
                                const void* drafter_comp_logits,
                                int dtype,
                                const int32_t* vocab_map, int Vd,
                                const int32_t* draft_tokens,
                                const float* draft_probs,
                                const float* uniforms,
                                const float* temperature,
                                int B, int K, int V,
                                const asymspec_params* params,
                                int32_t* accept_len,
                                int32_t* next_token,
                                float* fused_logprobs,
                                float* gate_out,
                                float* fused_logprobs_full,
                                void* workspace, size_t workspace_bytes,
                                void* stream);

/* ---- the same step without a caller workspace ------------------------- */
#define ASYMSPEC_NOALLOC_MAX_WORKSPACE (48u << 20)  /* bytes of static scratch per device */

/*
 * For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): asymspec_fuse_verify with
 * every argument but the workspace, which is instead a static device array
 * of ASYMSPEC_NOALLOC_MAX_WORKSPACE bytes that the library holds on each
 * device it runs on, for the life of the process.  No device memory is
 * allocated or freed by this call.
 *   - Shapes whose asymspec_workspace_size exceeds the array return
 *     ASYMSPEC_E_WORKSPACE with nothing enqueued (B = 512, K = 8, V = 256000
 *     bf16 needs 32.4 MiB and fits).
 *   - Every call on one device uses that device's array: calls that may
 *     overlap on one device (other streams, other host threads) race and
 *     must not be issued; calls in one stream are ordered and safe.
 *   - Nothing in the array must start at zero: every record the kernel
 *     exchanges carries the call's epoch.  Its timeout counter is read with
 *     asymspec_noalloc_timeouts (cumulative over the process).
 *   - The epoch is still a launch argument chosen here at each call, so a
 *     captured call must not be replayed (see asymspec_workspace_size).
 * Returns the status codes of asymspec_fuse_verify, or ASYMSPEC_E_DEVICE
 * when the array's device address cannot be found.
 */
int asymspec_fuse_verify_noalloc(const void* verifier_logits,
                                 const void* drafter_full_logits,
                                 const void* drafter_comp_logits,
                                 int dtype,
                                 const int32_t* draft_tokens,
                                 const float* draft_probs,
                                 const float* uniforms,
                                 const float* temperature,
                                 int B, int K, int V,
                                 const asymspec_params* params,
                                 int32_t* accept_len,
                                 int32_t* next_token,
                                 float* fused_logprobs,
                                 float* gate_out,
                                 float* fused_logprobs_full,
                                 void* stream);

/* Timed-out waits counted in the current device's static array (see
 * asymspec_workspace_timeouts; synchronises `stream`). */
int asymspec_noalloc_timeouts(void* stream, uint32_t* count);

/* Number of timed-out waits between workgroups recorded in `workspace`
 * since it was last zero-filled (asymspec_workspace_clear, or a zeroed
 * allocation), into *count (a host pointer).  The decision kernel's
 * workgroups exchange records through the workspace; every wait for one is
 * bounded (0.2 s by default, asymspec_set_wait_limit), and a wait that runs
 * out is counted here.  A request whose decision could not be completed has
 * accept_len = -1 and unspecified other outputs; every other request's
 * outputs are valid.  A nonzero count means the device did not run the
 * launch's workgroups as the kernel assumes (for example calls sharing one
 * workspace overlapped) and should be treated as an error.
 *   workspace        the workspace passed to the calls (device pointer,
 *                    256-byte aligned, at least 256 bytes)
 *   stream           the stream the calls were enqueued on: the count is read
 *                    after every call enqueued before this one (the call
 *                    synchronises the stream)
 * Returns ASYMSPEC_OK, ASYMSPEC_E_ARG or ASYMSPEC_E_DEVICE. */
int asymspec_workspace_timeouts(const void* workspace, size_t workspace_bytes, void* stream,
                                uint32_t* count);

/* Sets the bound of every wait between workgroups for calls enqueued after
 * it, process-wide, in ticks of the GPU's 100 MHz clock (10 ns each); 0
 * restores the default of 20,000,000 (0.2 s); at most 100,000,000 (1 s),
 * else ASYMSPEC_E_ARG.  A test hook for the error path: a bound of a few
 * ticks makes waits run out under normal operation, and every workgroup
 * still ends. */
int asymspec_set_wait_limit(unsigned long long ticks);

/* Static text for a status code. */
const char* asymspec_status_string(int status);

/* Library version, major * 10000 + minor * 100 + patch. */
int asymspec_version(void);

#ifdef __cplusplus
}
#endif
#endif /* ASYMSPEC_H */
