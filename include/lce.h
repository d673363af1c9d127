/*
 * lce.h -- C ABI of the MI355X (gfx950) linear-cross-entropy library, liblce.so.
 *
 * The objective (paper Sec. 4.2, "Linear Cross-Entropy loss"): fuse the model's
 * final output projection with the cross-entropy over the whole vocabulary,
 * drop ignored target positions before the projection, and never hold the
 * [tokens, vocab] logit matrix. It is a drop-in for the standard cross-entropy
 * objective (Sec. 3.3), so for hidden states H [N, D], projection weight
 * W [V, D] (the nn.Linear(D, V) weight) and targets t [N]:
 *
 *   M   = { n : t_n != ignore_index and 0 <= t_n < V },  Nv = |M|
 *   s   = H W^T (per row; never stored whole)
 *   lse_n = log sum_v exp(s[n, v]),   l_n = lse_n - s[n, t_n]            (n in M)
 *   L   = (1/Nv) sum_{n in M} l_n  (mean),  sum_{n in M} l_n  (sum),
 *         or the per-token vector l_n, 0 outside M  (none: minus the per-token
 *         log-probability of the target, the quantity DPO / GRPO style losses consume)
 *   G   = c_n (softmax(s) - onehot(t)) on rows in M, 0 elsewhere;
 *         c_n = g/Nv (mean), g (sum) or g_n (none, one upstream gradient per token)
 *   dH  = G W,   dW = G^T H
 *
 * Conventions shared by every entry point
 *  - All tensors are caller-owned device memory; the library never allocates
 *    device memory and keeps no state between calls. The one exception is the
 *    optional kernel-timing facility below, the library's only mutable global
 *    state: a process-wide pool of HIP events behind a mutex, used for profiling.
 *  - H, W, dH and dW are bf16 (stored as 16-bit words), row-major. H and W may
 *    have a row stride (ld_h, ld_w, in elements, >= d, multiple of 8); dH and dW
 *    are dense [N, D] and [V, D]. Every pointer must be 16-byte aligned; the
 *    workspace must be 256-byte aligned. d must be a multiple of 8.
 *  - targets are int32 (target_bytes = 4) or int64 (target_bytes = 8).
 *  - Outputs must not alias inputs.
 *  - Calls only enqueue work on `stream` (a hipStream_t; NULL = the default
 *    stream): no host synchronisation and no allocation, so a forward/backward
 *    pair can be captured in a HIP graph. The workspace may be reused as soon
 *    as the stream has finished the call.
 *  - Host-detectable errors (null pointers, bad sizes, misalignment, small
 *    workspace) are returned before anything is launched. A failed launch
 *    returns LCE_ERR_HIP. Bad target values are data, seen only on the device:
 *    such rows are treated as ignored and bit 0 of *dev_status is set.
 *  - Results are deterministic: the same inputs give the same bits on every run
 *    (no atomics in any reduction; fixed summation orders).
 */
#ifndef LCE_H_
#define LCE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum lce_status {
  LCE_OK = 0,
  LCE_ERR_NULL = 1,         /* a required pointer is NULL */
  LCE_ERR_SHAPE = 2,        /* n < 0, d < 1, v < 1, ld < d, or sizes beyond 32-bit offsets */
  LCE_ERR_ALIGN = 3,        /* pointer, stride or workspace misaligned */
  LCE_ERR_UNSUPPORTED = 4,  /* d % 8 != 0, unknown reduction or target width */
  LCE_ERR_WORKSPACE = 5,    /* workspace smaller than lce_workspace_size() */
  LCE_ERR_HIP = 6,          /* a HIP runtime call or kernel launch failed */
  LCE_ERR_ARG = 7           /* other invalid argument */
} lce_status_t;

typedef enum lce_reduction {
  LCE_REDUCE_MEAN = 0,      /* divide by the valid-token count Nv of this call */
  LCE_REDUCE_SUM = 1,
  LCE_REDUCE_NONE = 2       /* per-token losses; loss and grad_loss are [N] arrays */
} lce_reduction_t;

/* Bit set in *dev_status by lce_forward when some target is neither ignore_index nor in [0, V). */
#define LCE_STATUS_TARGET_OUT_OF_RANGE 1

typedef struct lce_problem {
  int64_t n;                /* tokens (rows of H, entries of targets) */
  int64_t d;                /* hidden size (multiple of 8) */
  int64_t v;                /* vocabulary size (rows of W), >= 1 */
  int64_t ld_h;             /* row stride of H in elements; 0 means d */
  int64_t ld_w;             /* row stride of W in elements; 0 means d */
  int32_t ignore_index;     /* targets equal to this are ignored (e.g. -100) */
  int32_t reduction;        /* lce_reduction_t */
  int32_t target_bytes;     /* 4 (int32 targets) or 8 (int64 targets) */
  int32_t flags;            /* bitwise OR of LCE_FLAG_* (0 for none); unknown bits are rejected */
} lce_problem_t;

/* lce_backward adds this call's dW to the values already in dW instead of overwriting it:
 * dW = bf16(float(dW) + fp32 contribution). This is gradient accumulation over micro-batches,
 * which the paper's benchmark settings use (performance benchmarks) and which its Sec. 4.1
 * names as the case the fused optimizer step cannot serve. lce_forward ignores the flag;
 * lce_backward_adamw rejects it (one update per backward pass). */
#define LCE_FLAG_ACCUMULATE_DW 1

/* For lce_backward, lce_backward_adamw and lce_backward_shard: the workspace still holds what the
 * immediately preceding lce_forward (or lce_forward_shard, then lce_combine_shards) of the same
 * problem, H and targets left in it, on the same stream and with nothing else written to the
 * workspace in between. The backward then reuses that call's valid-row list (and, where the
 * forward gathered them, the valid rows of H) instead of forming them again: two fewer kernels
 * per step. Without the flag the backward depends on no earlier call. The forward and the
 * combine ignore the flag; the KD calls reject it (LCE_ERR_ARG). The workspace must be at
 * least max(fwd_bytes, bwd_bytes). */
#define LCE_FLAG_REUSE_FORWARD 2

/*
 * Hyper-parameters of one AdamW step (decoupled weight decay, bias-corrected moments), the
 * optimizer that paper Sec. 4.1 fuses into the backward pass. With t = step:
 *   theta <- theta (1 - lr weight_decay)
 *   m <- beta1 m + (1 - beta1) g,     v <- beta2 v + (1 - beta2) g^2
 *   theta <- theta - lr / (1 - beta1^t) * m / (sqrt(v) / sqrt(1 - beta2^t) + eps)
 * The constants are formed on the host in double precision and used in fp32 on the device.
 */
typedef struct lce_adamw {
  float lr;                 /* >= 0 */
  float beta1, beta2;       /* in [0, 1) */
  float eps;                /* >= 0 */
  float weight_decay;       /* >= 0 */
  int32_t step;             /* t >= 1: the 1-based index of this update */
  int32_t reserved;         /* must be 0 */
} lce_adamw_t;

/*
 * Workspace sizes, in bytes, for lce_forward (*fwd_bytes) and lce_backward
 * (*bwd_bytes). They grow as O(N*D + N*V_slab) with V_slab = max(8192, 4*D, Vw)
 * rounded up to a multiple of 6144 (at most V rounded up to 768), Vw = min(24576,
 * 160 MiB / (2*D) rounded down to 6144), or, where it gives the dW launches fewer
 * workgroup rounds, another multiple of 768 between max(8192, 4*D) and
 * min(24576, 160 MiB / (2*D)) (lce_plan_info reports the width): never O(N*V).
 * The backward's size does not depend on V; the forward's vocabulary partials
 * take at most 2*D bytes per token. Either output pointer may be NULL.
 */
lce_status_t lce_workspace_size(const lce_problem_t* p, size_t* fwd_bytes, size_t* bwd_bytes);

/*
 * Layout of the workspace that lce_forward and lce_backward carve for problem p, for tests and
 * tools that check it (host only; nothing is launched). Offsets and sizes are in bytes from the
 * workspace start; rows in elements. A prefix is shared by both passes: the valid-row list idx
 * and inverse map pos ([npad] int32 each), the count Nv, and the gathered valid rows of H
 * ([npad][d] bf16). The forward then holds its vocabulary partial pairs (two [part_rows][npad]
 * fp32 arrays) and per-row terms ([npad] fp32); the backward holds G ([rows_g][vc] bf16, one
 * vocabulary slab of vc ids, nslab slabs) and the fp32 dH accumulators: dh_kz of them, [rows_g][d]
 * each, one after the other from o_dh32, when the dH launches split K into dh_kz parts (launches
 * with fewer output tiles than compute units; o_dh32b is the second one's offset, or 0). With
 * dh_kz = 1 the launches split the K range of the tiles of each XCD's last partial round on the
 * device, and keep those parts in the accumulator's rows past the valid ones.
 */
typedef struct lce_plan_info {
  int64_t npad;             /* N rounded up to 256 */
  int64_t rows_g;           /* npad rounded up to 384: rows of G and of the dH accumulators */
  int64_t vc, nslab;        /* backward slab width (ids) and slab count */
  int64_t dh_kz;            /* K parts of the dH launches: 1, or up to 8 for launches with few tiles */
  int64_t part_rows;        /* partial rows of the forward statistics */
  int64_t fwd_gathers;      /* 1 if the forward leaves the gathered rows of H in the prefix */
  int64_t fwd_one_launch;   /* 1 if the forward statistics run as one launch */
  int64_t o_idx, o_pos, o_nv, o_hv;
  int64_t o_pm, o_ps, o_terms, fwd_bytes;
  int64_t o_g, o_dh32, o_dh32b, bwd_bytes;
} lce_plan_info_t;

lce_status_t lce_plan_info(const lce_problem_t* p, lce_plan_info_t* out);

/*
 * Forward pass (paper Sec. 4.2): computes the loss without materialising the
 * logits. Outputs, all device memory:
 *   loss        fp32: [1] L for mean / sum (0 when Nv = 0); [N] per-token losses
 *               for LCE_REDUCE_NONE (0.0 on ignored / bad rows)
 *   lse         [N] fp32: lse_n for valid rows, 0.0 for ignored / bad rows;
 *               keep it for lce_backward
 *   n_valid     [1] int32: Nv
 *   dev_status  [1] int32 or NULL: overwritten with status bits
 *               (LCE_STATUS_TARGET_OUT_OF_RANGE)
 */
lce_status_t lce_forward(const lce_problem_t* p,
                         const void* H, const void* W, const void* targets,
                         float* loss, float* lse, int32_t* n_valid, int32_t* dev_status,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * Backward pass of the same objective (paper Sec. 4.2; the gradients of the standard
 * cross-entropy it replaces, Sec. 3.3): recomputes the logits tile by tile (they were never
 * stored), forms G = c (softmax - onehot) one vocabulary slab at a time and writes both
 * gradients, dH = G W and dW = G^T H.
 *   lse         [N] fp32 from lce_forward on the same inputs
 *   n_valid     [1] int32: the count that "mean" divides by (lce_forward's
 *               n_valid on one device; a global count when the tokens of one
 *               batch are spread over several calls); unused for NONE
 *   grad_loss   fp32, read on the device: [1] upstream gradient g of L for mean /
 *               sum; [N] upstream gradients g_n of the per-token losses for NONE
 *   dH          [N, D] bf16, overwritten; rows of ignored tokens are +0.0
 *   dW          [V, D] bf16, overwritten (or added to, with LCE_FLAG_ACCUMULATE_DW)
 */
lce_status_t lce_backward(const lce_problem_t* p,
                          const void* H, const void* W, const void* targets,
                          const float* lse, const int32_t* n_valid, const float* grad_loss,
                          void* dH, void* dW,
                          void* workspace, size_t workspace_bytes, void* stream);

/*
 * lce_forward for callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): the same computation and outputs as
 * lce_forward, bit for bit, with the workspace taken from a fixed device array inside the library
 * instead of from the caller. The array holds LCE_NOALLOC_SCRATCH_BYTES (256 MiB) on every GPU
 * the library runs on, from the first call on that GPU until the process ends; problems whose
 * forward workspace (lce_workspace_size's fwd_bytes) is larger are rejected with
 * LCE_ERR_WORKSPACE before anything is launched. The call itself allocates nothing. All calls on
 * one GPU share its array: calls that may overlap on one GPU (on different streams, or from
 * several threads onto different streams) race and must be ordered by the caller; calls on one
 * stream are ordered by it. `stream` must belong to the current device (else LCE_ERR_ARG). The
 * backward of a problem forwarded this way is lce_backward with a workspace of its own.
 */
#define LCE_NOALLOC_SCRATCH_BYTES (256u * 1024u * 1024u)
lce_status_t lce_forward_noalloc(const lce_problem_t* p,
                                 const void* H, const void* W, const void* targets,
                                 float* loss, float* lse, int32_t* n_valid, int32_t* dev_status,
                                 void* stream);

/*
 * Two-phase optimizer step (the standard path that in-backward fusion replaces, paper Sec.
 * 4.1): one AdamW step on the bf16 parameter W [V, D] (row stride ld_w, 0 means d) with the
 * bf16 gradient dW [V, D] (dense, as lce_backward writes it; NULL means a zero gradient).
 *   exp_avg, exp_avg_sq  [V, D] fp32, dense, updated in place (start at 0 for step 1)
 *   W_master             [V, D] fp32 or NULL. If given, it is the parameter: it is updated and
 *                        W receives its bf16 rounding (nearest, ties to even). If NULL, the
 *                        parameter is W itself, read as fp32 and rounded back to bf16.
 * Element by element the arithmetic is exactly that of lce_backward_adamw, so the two paths
 * give the same bits. All pointers 16-byte aligned; v >= 1, d >= 8 and a multiple of 8.
 */
lce_status_t lce_adamw_step(int64_t v, int64_t d, int64_t ld_w, void* W, const void* dW,
                            float* exp_avg, float* exp_avg_sq, float* W_master,
                            const lce_adamw_t* opt, void* stream);

/*
 * Backward pass with the optimizer step fused in (paper Sec. 4.1 applied to the LCE weight of
 * Sec. 4.2): as lce_backward, but instead of writing dW, each vocabulary slab's dW block
 * (rounded to bf16 exactly as lce_backward would store it) is consumed at once by an AdamW step
 * on that slab of W, so no [V, D] gradient buffer ever exists. W, exp_avg, exp_avg_sq and
 * W_master are as in lce_adamw_step and are updated in place; dH is written as by
 * lce_backward (it uses the weights from before the step). The result is bitwise identical to
 * lce_backward followed by lce_adamw_step with the same opt. W must not be read or written by
 * other work while the call runs. p->flags must not contain LCE_FLAG_ACCUMULATE_DW. The
 * workspace is lce_backward's (bwd_bytes).
 */
lce_status_t lce_backward_adamw(const lce_problem_t* p,
                                const void* H, void* W, const void* targets,
                                const float* lse, const int32_t* n_valid, const float* grad_loss,
                                void* dH, float* exp_avg, float* exp_avg_sq, float* W_master,
                                const lce_adamw_t* opt,
                                void* workspace, size_t workspace_bytes, void* stream);

/*
 * Vocabulary-parallel ("loss parallel") mode. The paper composes the loss with loss-parallel
 * sharding of the output projection over the vocabulary (Sec. 4.2, Sec. 5): each of G shards
 * holds the rows of W for ids [v_begin, v_begin + p->v) of a vocabulary of v_total ids. Then
 *   lse_n = log sum_g exp(lse_n^g)       (lse_n^g: log-sum-exp over shard g's ids)
 *   s[n, t_n] = sum_g tgt_n^g            (tgt_n^g: the target logit if shard g holds t_n, else 0)
 * so a forward needs only O(N) numbers per shard, and each shard's backward, given the global
 * lse, yields its rows of dW and its term G_g W_g of dH (the terms sum to dH).
 * The collectives that move these numbers between devices belong to the caller: gather the
 * [N] partials of every shard into [G, N] arrays for lce_combine_shards, and sum the dH terms.
 */
typedef struct lce_shard {
  int64_t v_total;          /* ids of the whole vocabulary; targets are ids in [0, v_total) */
  int64_t v_begin;          /* first id of this shard: W row r is id v_begin + r */
} lce_shard_t;

/*
 * Forward of one shard (p->v = rows of this shard; p->reduction is not used). Outputs:
 *   lse_part  [N] fp32: log-sum-exp over this shard's ids for valid rows, 0.0 elsewhere
 *   tgt_part  [N] fp32: s[n, t_n] if this shard holds t_n, else 0.0
 *   n_valid, dev_status as lce_forward (validity is judged against v_total)
 * Workspace: lce_workspace_size(p) forward bytes. Errors: LCE_ERR_SHAPE if the shard range is
 * not inside [0, v_total) or v_total >= 2^30.
 */
lce_status_t lce_forward_shard(const lce_problem_t* p, const lce_shard_t* shard,
                               const void* H, const void* W, const void* targets,
                               float* lse_part, float* tgt_part, int32_t* n_valid, int32_t* dev_status,
                               void* workspace, size_t workspace_bytes, void* stream);

/*
 * Combine of G = n_shards shards' partials into the full-vocabulary results (p->v = v_total;
 * p->d is checked as elsewhere but not used). lse_parts and tgt_parts are [G, N] fp32, row g
 * holding shard g's lse_part / tgt_part (any shard order). Outputs loss, lse, n_valid and
 * dev_status exactly as lce_forward defines them. The combine runs over shards in row order,
 * so every device that combines the same arrays gets the same bits. 1 <= n_shards <= 4096.
 * Workspace: lce_workspace_size(p) forward bytes.
 */
lce_status_t lce_combine_shards(const lce_problem_t* p, int32_t n_shards,
                                const float* lse_parts, const float* tgt_parts, const void* targets,
                                float* loss, float* lse, int32_t* n_valid, int32_t* dev_status,
                                void* workspace, size_t workspace_bytes, void* stream);

/*
 * Backward of one shard, given the full-vocabulary lse (from lce_combine_shards) and the global
 * n_valid: G_g = c (exp(s - lse) - onehot) over this shard's ids (onehot only where the shard
 * holds the target).
 *   dH_part   [N, D] fp32 dense, overwritten: G_g W_g (rows of invalid tokens 0.0); the sum over
 *             shards is dH, kept in fp32 so that the sum loses nothing to bf16 rounding
 *   dW        [p->v, D] bf16 dense: this shard's rows of dW (LCE_FLAG_ACCUMULATE_DW applies)
 * Workspace: lce_workspace_size(p) backward bytes.
 */
lce_status_t lce_backward_shard(const lce_problem_t* p, const lce_shard_t* shard,
                                const void* H, const void* W, const void* targets,
                                const float* lse, const int32_t* n_valid, const float* grad_loss,
                                float* dH_part, void* dW,
                                void* workspace, size_t workspace_bytes, void* stream);

/*
 * Fused linear knowledge-distillation loss. The paper's recipes include knowledge distillation
 * with dedicated KD losses (Sec. 3.2, after Hinton et al., cited in Sec. 2); here it is built on
 * the LCE tiling for a student head (Hs [N, Ds], Ws [V, Ds]) and a teacher head (Ht [N, Dt],
 * Wt [V, Dt]) over the same tokens and vocabulary, with temperature T:
 *   p_t = softmax(Ht Wt^T / T),  zs = Hs Ws^T / T
 *   l_n = lse(zs_n) - sum_v p_t(v) zs_n(v)       soft-target cross-entropy, n in M
 *   L   = mean / sum over M, or the per-token l_n (0 outside M), as for lce_forward
 *   G   = c (softmax(zs) - p_t) / T,  dHs = G Ws,  dWs = G^T Hs     (no teacher gradient)
 * Labels only define the valid set M (as for LCE: not ignore_index and in [0, V)). The loss
 * is not multiplied by T^2; neither logit matrix is ever held whole (the teacher's
 * probabilities exist one vocabulary slab at a time, in the workspace).
 */
typedef struct lce_kd_problem {
  int64_t n;                /* tokens */
  int64_t ds, dt;           /* student / teacher hidden sizes (multiples of 8) */
  int64_t v;                /* vocabulary size shared by both heads */
  int64_t ld_hs, ld_ws, ld_ht, ld_wt;   /* row strides in elements; 0 means dense */
  float temperature;        /* T > 0 */
  int32_t ignore_index;
  int32_t reduction;        /* lce_reduction_t */
  int32_t target_bytes;     /* 4 or 8 */
  int32_t flags;            /* LCE_FLAG_ACCUMULATE_DW applies to dWs */
  int32_t reserved;         /* must be 0 */
} lce_kd_problem_t;

/* Workspace bytes of lce_kd_forward / lce_kd_backward: O(N (Ds + Dt) + N V_slab) with the
 * student's slab width, never O(N V). */
lce_status_t lce_kd_workspace_size(const lce_kd_problem_t* p, size_t* fwd_bytes, size_t* bwd_bytes);

/*
 * KD forward. Outputs (device): loss ([1], or [N] per token for LCE_REDUCE_NONE), lse_s and
 * lse_t ([N] fp32: log-sum-exp of zs and of the teacher's logits / T on valid rows, 0.0
 * elsewhere; keep both for the backward), n_valid, dev_status (nullable) as for lce_forward.
 */
lce_status_t lce_kd_forward(const lce_kd_problem_t* p,
                            const void* Hs, const void* Ws, const void* Ht, const void* Wt,
                            const void* targets, float* loss, float* lse_s, float* lse_t,
                            int32_t* n_valid, int32_t* dev_status,
                            void* workspace, size_t workspace_bytes, void* stream);

/*
 * KD backward: dHs [N, Ds] bf16 (overwritten, 0 on rows outside M) and dWs [V, Ds] bf16
 * (overwritten, or added to with LCE_FLAG_ACCUMULATE_DW); grad_loss and n_valid as for
 * lce_backward; lse_s / lse_t from lce_kd_forward on the same inputs.
 */
lce_status_t lce_kd_backward(const lce_kd_problem_t* p,
                             const void* Hs, const void* Ws, const void* Ht, const void* Wt,
                             const void* targets, const float* lse_s, const float* lse_t,
                             const int32_t* n_valid, const float* grad_loss, void* dHs, void* dWs,
                             void* workspace, size_t workspace_bytes, void* stream);

/*
 * KD forward and backward in one call, for the usual case where the KD loss is the objective
 * being differentiated: grad_loss is read on the device when the gradient kernels run. The
 * teacher's probabilities are formed once per slab (not once in the forward and again in the
 * backward) and one student pass per slab yields both G and the loss's partial sums, so the MFMA
 * work is 4 Nv V Dt + 8 Nv V Ds instead of 6 Nv V Dt + 10 Nv V Ds. Outputs are those of
 * lce_kd_forward and lce_kd_backward, bit for bit. Workspace: lce_kd_workspace_size_fused.
 */
lce_status_t lce_kd_workspace_size_fused(const lce_kd_problem_t* p, size_t* bytes);
lce_status_t lce_kd_forward_backward(const lce_kd_problem_t* p,
                                     const void* Hs, const void* Ws, const void* Ht, const void* Wt,
                                     const void* targets, const float* grad_loss,
                                     float* loss, float* lse_s, float* lse_t,
                                     int32_t* n_valid, int32_t* dev_status, void* dHs, void* dWs,
                                     void* workspace, size_t workspace_bytes, void* stream);

/* Static, human-readable name of a status code. */
const char* lce_status_string(lce_status_t s);

/*
 * Optional per-kernel timing, for profiling only. When enabled, every kernel
 * launch of the calls above is bracketed by a pair of HIP events recorded on
 * the caller's stream (up to a fixed pool of pairs per enable; later launches
 * are not recorded). lce_timing_read waits for the recorded events and
 * returns the summed milliseconds and the number of launches of kernel `k`
 * (0 <= k < lce_timing_kernel_count()). Enabling resets the records. The pool
 * (8192 event pairs, created on the first enable on the current device and kept
 * until the process ends) and the on/off switch are global to the process and
 * guarded by a mutex; they are the library's only mutable global state, and the
 * compute entry points touch them only while timing is on. Enabling creates HIP
 * events, so these calls are not for graph capture.
 */
lce_status_t lce_timing_enable(int on);
int lce_timing_kernel_count(void);
const char* lce_timing_kernel_name(int k);
lce_status_t lce_timing_read(int k, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* LCE_H_ */
