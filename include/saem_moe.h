/*
 * saem_moe.h -- C ABI of libsaem_moe.so: one MoE layer's forward on MI355X (gfx950).
 *
 * The operations follow SAEM (arXiv 2608.21614):
 *   - top-k gating by a router (Section II-A);
 *   - expert-aligned token repacking: the (token, expert) pairs of a batch are
 *     grouped by expert into contiguous buffers, using only index reordering
 *     and a workspace allocated once and reused across layers (Section IV-E.1,
 *     Section VI-A);
 *   - partition of the repacked batch by the residency map into GPU-bound rows
 *     and a packed list of host-bound rows (Section IV-D.2), over a fixed set of
 *     per-layer expert slots (Section IV-C.1, IV-C.2);
 *   - one batched execution per resident expert (Section IV-E.1) on the matrix
 *     cores (Section IV-D.2);
 *   - a merge of the expert outputs back to token order (Section IV-D.2).
 * The expert MLP is SwiGLU without biases: y = (silu(x W1) * (x W3)) W2.
 *
 * Conventions for every call
 *   - Returns moe_status.  No exception or abort crosses the ABI.
 *   - All tensor pointers are DEVICE pointers owned by the caller (except for
 *     the host-side calls moe_stage_plan, moe_host_ffn and moe_offload_plan).  The library never
 *     allocates or frees device memory and never synchronises the stream.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL is the null stream).
 *   - Arguments are validated on the host before anything is enqueued; a call
 *     that returns an error has enqueued nothing.  Validation never touches
 *     device memory, so it works on a machine without a GPU.
 *   - Kernel faults surface at the caller's next synchronisation, as usual for
 *     HIP; launch failures return MOE_ERR_HIP.
 *   - Calls on distinct streams with distinct workspaces may run concurrently.
 *   - Alignment (MOE_ERR_INVALID_ARG otherwise): activations, weights, outputs,
 *     y, y_off, off_rows and the workspace 16 bytes; index, count, slot, score
 *     and gate arrays 4 bytes; the int64 stage log 8 bytes.
 *   - Layouts:
 *       x          [T, H]        activations (dims.dtype), row-major
 *       w_router   [E, H]        row e scores expert e (dims.dtype), row-major
 *       bias       [E]           fp32 router bias, or NULL
 *       w13        [slots, 2F, H] per slot, in the TILE LAYOUT (moe_pack_weights):
 *                                logical rows 0..F-1 are the gate projection W1
 *                                (row f = output feature f), rows F..2F-1 the
 *                                up projection W3, K = H
 *       w2         [slots, H, F] per slot, tile layout: row h = output feature h
 *                                of W2, K = F
 *       ws13, ws2  [S, 2Fs, H], [S, H, Fs] shared experts, same tile layout
 *     Tile layout of a logical [R, K] matrix: blocks of 16 rows x 32 columns;
 *     block (rt, s) starts at element (rt * K/32 + s) * 512 and its element
 *     8*l + i holds W[16*rt + l%16][32*s + 8*(l/16) + i].  Same size as the
 *     row-major matrix.
 *   - Residency map: expert_slot[E] (int32, device).  Expert e is resident iff
 *     0 <= expert_slot[e] < dims.slots, and then its weights are
 *     w13[expert_slot[e]] and w2[expert_slot[e]]; any other value (e.g. -1)
 *     means offloaded.  A slot holds one expert: two resident experts must not
 *     share a slot (the FFN may then run only one of them; nothing faults).
 *   - A routed pair q = t*k + j is the j-th selected expert of token t.
 *   - Packed rows: the pairs of resident experts first, experts in ascending id,
 *     then the pairs of offloaded experts, experts in ascending id; inside an
 *     expert, ascending token.  n_res = number of resident pairs, so rows
 *     [0, n_res) are GPU-bound and rows [n_res, T*k) form the offloaded list.
 */
#ifndef SAEM_MOE_H
#define SAEM_MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOE_ABI_VERSION 1

typedef enum moe_status {
    MOE_OK = 0,
    MOE_ERR_INVALID_ARG = 1,  /* NULL pointer, negative size, k > E, bad struct_size, ... */
    MOE_ERR_UNSUPPORTED = 2,  /* valid but not supported: H or F not a multiple of 64, E > 256, k > 8 */
    MOE_ERR_WORKSPACE = 3,    /* workspace NULL or smaller than moe_workspace_bytes() */
    MOE_ERR_HIP = 4,          /* a HIP launch or runtime call failed */
    MOE_ERR_SCRATCH_LIMIT = 5 /* moe_layer_forward_noalloc: the layer's workspace exceeds MOE_NOALLOC_SCRATCH_BYTES */
} moe_status;

typedef enum moe_dtype {
    MOE_F32 = 0,   /* IEEE fp32 */
    MOE_BF16 = 1   /* bfloat16 (fp32 accumulation everywhere) */
} moe_dtype;

/* Shapes of one MoE layer. */
typedef struct moe_dims {
    int32_t tokens;      /* T >= 0; T == 0 is a valid no-op that writes n_res = 0 */
    int32_t hidden;      /* H >= 64, multiple of 64 */
    int32_t experts;     /* E routed experts, 1..256 */
    int32_t ffn;         /* F >= 64, multiple of 64 (routed expert width) */
    int32_t top_k;       /* k, 1..min(E, 8) */
    int32_t shared;      /* S >= 0 always-on shared experts (at most 8) */
    int32_t shared_ffn;  /* Fs, multiple of 64 when S > 0, ignored when S == 0 */
    int32_t slots;       /* number of resident-expert slots held in w13 / w2, 0..E */
    int32_t dtype;       /* moe_dtype of x, w_router, w13, w2, ws13, ws2 */
} moe_dims;

/* flags of moe_route_topk and moe_layer_forward */
#define MOE_LOGITS_IN 1u   /* route the caller's scores in `logits`; x and w_router are not read */

int moe_abi_version(void);

/* Static description of a status code. */
const char* moe_status_str(moe_status s);

/* Host-only validation of a shape description. */
moe_status moe_check_dims(const moe_dims* dims);

/*
 * Bytes of workspace any call below needs for these dims (Section IV-E.1: the
 * repacking workspace is allocated once and reused across all MoE layers).
 * One workspace sized for the largest layer serves every call.
 */
moe_status moe_workspace_bytes(const moe_dims* dims, size_t* bytes);

/*
 * Router scores and top-k gate (Section II-A).
 *   logits  [T,E] fp32: written with x . w_router[e] + bias[e] (fp32
 *           accumulation), or, with MOE_LOGITS_IN, read as given (then x,
 *           w_router and bias are not used: the scores are final).
 *   topk_idx [T,k] int32: the k highest scores of each token in decreasing
 *           order; equal scores go to the lower expert id.
 *   topk_w  [T,k] fp32: softmax of the k selected scores (renormalised gate);
 *           a selected score equal to the top one contributes exactly 1, so a
 *           row of equal scores (also all -inf) gets 1/k.  NaN scores: undefined.
 *   ws:     workspace of moe_workspace_bytes(dims) bytes (partial scores).
 */
moe_status moe_route_topk(const moe_dims* dims, const void* x, const void* w_router, const float* bias,
                          float* logits, uint32_t flags, int32_t* topk_idx, float* topk_w, void* ws, size_t ws_bytes,
                          void* stream);

/*
 * Expert-aligned token repacking with the residency split (Section IV-E.1,
 * Section IV-D.2).
 *   in:  topk_idx [T,k] (ids outside [0,E) are dropped: no row, inv_perm = -1),
 *        topk_w [T,k] (read only if off_w != NULL), expert_slot [E],
 *        x [T,H] (read only if off_rows != NULL)
 *   out: counts [E]      pairs per expert
 *        seg_start [E]   first packed row of each expert
 *        perm [T*k]      pair q stored at packed row p (perm[p] = q)
 *        inv_perm [T*k]  packed row of pair q
 *        n_res [1]       resident pairs
 *        off_rows [T*k, H] (optional): off_rows[p - n_res] = x[perm[p] / k] for
 *                        the offloaded rows p in [n_res, T*k)
 *        off_w [T*k] (optional): the matching gate weights
 * n_res stays in device memory; the caller copies it (and the offloaded list)
 * to the host when it runs the offloaded experts there.
 */
moe_status moe_repack(const moe_dims* dims, const int32_t* topk_idx, const float* topk_w,
                      const int32_t* expert_slot, const void* x, int32_t* counts, int32_t* seg_start,
                      int32_t* perm, int32_t* inv_perm, int32_t* n_res, void* off_rows, float* off_w,
                      void* stream);

/*
 * Grouped SwiGLU expert FFN over the resident experts and the shared experts
 * (Section IV-D.2, Section IV-E.1): every resident expert with tokens runs once
 * over its packed rows; every shared expert runs over all T tokens.
 *   y [T*k + S*T, H] fp32: row p < T*k is packed row p (written for resident
 *     rows [0, n_res) only; the offloaded rows are left untouched for the
 *     host); row T*k + s*T + t is shared expert s on token t.
 * Counts and offsets are read from device memory: no host synchronisation.
 * ws13 / ws2 may be NULL when S == 0.
 */
moe_status moe_grouped_ffn(const moe_dims* dims, const void* x, const int32_t* perm, const int32_t* counts,
                           const int32_t* seg_start, const int32_t* expert_slot, const void* w13, const void* w2,
                           const void* ws13, const void* ws2, float* y, void* ws, size_t ws_bytes, void* stream);

/*
 * Merge back to token order (Section IV-D.2), deterministic: for each token,
 * in this fixed order and accumulated in fp32,
 *   out[t] = sum_j w[t,j] * y[inv_perm[t*k+j]]        (resident experts)
 *          + sum_j w[t,j] * y_off[inv_perm[t*k+j] - n_res]  (offloaded, only if y_off)
 *          + sum_s y[T*k + s*T + t]                     (shared experts)
 * then rounded once to out_dtype (MOE_F32, or MOE_BF16 with round-to-nearest-even).
 *   y_off [T*k - n_res, H] fp32: the host's outputs for the offloaded list, in
 *     packed order, or NULL for the resident-plus-shared partial.
 *   n_res: device pointer, read only if y_off != NULL.
 */
moe_status moe_combine(const moe_dims* dims, const int32_t* topk_idx, const float* topk_w,
                       const int32_t* inv_perm, const int32_t* expert_slot, const float* y,
                       const float* y_off, const int32_t* n_res, void* out, int32_t out_dtype, void* stream);

/* Arguments of the fused layer forward. */
typedef struct moe_layer_args {
    size_t struct_size;          /* sizeof(moe_layer_args) */
    moe_dims dims;
    uint32_t flags;              /* MOE_LOGITS_IN */
    int32_t out_dtype;           /* MOE_F32 or dims.dtype */
    const void* x;               /* [T,H] (not read with MOE_LOGITS_IN except for shared experts, FFN and off_rows) */
    const void* w_router;        /* [E,H] (not read with MOE_LOGITS_IN) */
    const float* bias;           /* [E] or NULL */
    const int32_t* expert_slot;  /* [E] */
    const void* w13;             /* [slots, 2F, H] */
    const void* w2;              /* [slots, H, F] */
    const void* ws13;            /* [S, 2Fs, H] or NULL if S == 0 */
    const void* ws2;             /* [S, H, Fs] or NULL if S == 0 */
    void* out;                   /* [T,H] out_dtype: resident + shared partial output */
    /* optional outputs; NULL keeps them in the workspace */
    float* logits;               /* [T,E]; required input with MOE_LOGITS_IN */
    int32_t* topk_idx;           /* [T,k] */
    float* topk_w;               /* [T,k] */
    int32_t* counts;             /* [E] */
    int32_t* seg_start;          /* [E] */
    int32_t* perm;               /* [T*k] */
    int32_t* inv_perm;           /* [T*k] */
    int32_t* n_res;              /* [1] */
    void* off_rows;              /* [T*k, H] dims.dtype, packed offloaded rows */
    float* off_w;                /* [T*k] */
    /* optional stage timing: NULL, or MOE_STAGE_EVENTS hipEvent_t handles the
     * caller created (timing enabled); the call records them on `stream`:
     * [0] before routing, [1] after routing, [2] after repacking, [3] after the
     * offloaded-row pack, [4] after FFN phase 1 (gate/up + SwiGLU), [5] after
     * FFN phase 2 (down projection), [6] after the combine.  At decode (T <= 64)
     * the repacking runs inside FFN phase 1 and the pack inside phase 2, so [2]
     * and [3] follow [1] directly. */
    void* const* stage_events;
} moe_layer_args;

#define MOE_STAGE_EVENTS 7

/*
 * Fused forward of one MoE layer: route -> repack (+ offloaded pack) ->
 * grouped SwiGLU FFN over resident and shared experts -> combine (at decode the
 * repacking and the pack run inside the two FFN launches).  `out` holds
 * the resident-plus-shared output; the offloaded list (off_rows, off_w,
 * perm[n_res:], n_res) is returned for host execution, whose results the caller
 * merges with moe_combine(..., y_off, ...).  Needs moe_workspace_bytes(&dims).
 */
moe_status moe_layer_forward(const moe_layer_args* args, void* ws, size_t ws_bytes, void* stream);

/* Size of the fixed device array that moe_layer_forward_noalloc uses as its workspace. */
#define MOE_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

/*
 * moe_layer_forward without a caller workspace and without any allocation, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc).  The workspace is a
 * fixed array of MOE_NOALLOC_SCRATCH_BYTES in the library, one per GPU, held
 * until the process ends; the caller still passes every input and output in
 * `args`, exactly as for moe_layer_forward, and gets the same results.
 *   - Layers whose moe_workspace_bytes() exceeds MOE_NOALLOC_SCRATCH_BYTES (in
 *     practice prefill-size batches) return MOE_ERR_SCRATCH_LIMIT, nothing enqueued.
 *   - `stream` must belong to the calling thread's current device (NULL: its
 *     null stream); a stream of another device returns MOE_ERR_INVALID_ARG.
 *   - The first call on a device looks up that device's array (no allocation).
 *   - All calls on one GPU share its array, and each leaves its intermediates
 *     there: calls that may overlap on one GPU (several streams, or threads)
 *     race on it and must be ordered by the caller.  Nothing is carried over
 *     from one call to the next.
 * Other errors as for moe_layer_forward.
 */
moe_status moe_layer_forward_noalloc(const moe_layer_args* args, void* stream);

/*
 * Converts one row-major [rows, cols] expert matrix (cols contiguous) into the
 * tile layout the FFN reads (see Layouts above).  Run once per expert when its
 * weights are placed in a slot (fixed per-layer expert slots, Section IV-C.1);
 * e.g. w13[slot] from the [2F, H] matrix whose row f is W1[:, f] and row F+f is
 * W3[:, f], and w2[slot] from the [H, F] matrix whose row h is W2[:, h].
 *   src, dst: device, distinct, rows * cols elements of `dtype` each.
 *   rows % 16 == 0 and cols % 32 == 0, else MOE_ERR_UNSUPPORTED.
 */
moe_status moe_pack_weights(const void* src, void* dst, int64_t rows, int64_t cols, int32_t dtype, void* stream);

/*
 * Stage-aware residency support (Section IV-B.2, Section IV-C.2).
 * moe_stage_accumulate adds a layer call's per-expert counts into an int64
 * activation log on the device: log[e] += counts[e].
 */
moe_status moe_stage_accumulate(int32_t experts, const int32_t* counts, int64_t* log, void* stream);

/*
 * Host-side residency plan at a stage boundary (Section IV-C.2): rank the
 * experts by the completed stage's activation count (ties: lower id first),
 * keep the top `slots`; an expert that stays keeps its slot, incoming experts
 * take the freed slots (by rank, freed slots in ascending order).
 *   log [E] (host), prev_slot [E] (host, -1 = offloaded) -> new_slot [E] (host).
 * Host memory only; no device work.
 */
moe_status moe_stage_plan(int32_t experts, int32_t slots, const int64_t* log, const int32_t* prev_slot,
                          int32_t* new_slot);

/* flags of moe_host_ffn */
#define MOE_HOST_PIN 1u    /* pin the worker threads to the calling thread's CPUs on one NUMA node */
#define MOE_HOST_NO_BF16_DOT 2u  /* bf16 layers: widen to fp32 in phase 1 even where the CPU has the
                                    AVX-512 bf16 dot-product instruction (used by default there) */

/*
 * In-situ host execution of the offloaded experts (Section IV-D.1, IV-D.2):
 * the SwiGLU of every offloaded expert over its rows of the packed offloaded
 * list, on the CPU, in parallel over output features, by `threads` worker
 * threads (<= 0: one per available CPU; with MOE_HOST_PIN, one per CPU of the
 * NUMA node).  The result is the y_off that moe_combine merges (the merge step
 * of Section IV-D.2).  Everything here is HOST memory; no device work.
 *   dims               the layer's shapes (dtype = dtype of the weights and rows)
 *   counts, seg_start  [E] int32, host copies of moe_repack's outputs
 *   n_res              host copy of moe_repack's n_res
 *   w13[e], w2[e]      host pointers, for every expert e with offloaded rows
 *                      (counts[e] > 0 and seg_start[e] >= n_res; others may be
 *                      NULL): ROW-MAJOR [2F, H] (rows 0..F-1 = W1, F..2F-1 =
 *                      W3) and [H, F] of dims.dtype, the matrices
 *                      moe_pack_weights takes for the device slots
 *   off_rows           [T*k - n_res, H] dims.dtype, host copy of the packed
 *                      offloaded rows (moe_repack / moe_layer_forward off_rows)
 *   y_off              [T*k - n_res, H] fp32 out: y_off[r] = SwiGLU_e(off_rows[r])
 *                      for the expert e that owns packed row n_res + r
 * fp32 accumulation; A = silu(x W1) * (x W3) is kept in fp32.  For bf16 layers
 * on a CPU with the AVX-512 bf16 dot-product instruction, x W1 and x W3 use it
 * (each bf16 product exact in fp32, pairs added into fp32 accumulators; inputs
 * below the fp32 normal range count as zero) unless flags has
 * MOE_HOST_NO_BF16_DOT.  Returns
 * MOE_ERR_INVALID_ARG if the offloaded segments do not tile [n_res, T*k) or a
 * needed pointer is NULL; nothing is written then.
 */
moe_status moe_host_ffn(const moe_dims* dims, const int32_t* counts, const int32_t* seg_start, int32_t n_res,
                        const void* const* w13, const void* const* w2, const void* off_rows, float* y_off,
                        int32_t threads, uint32_t flags);

/* Measured rates of the two ways to run an offloaded expert (moe_offload_plan). */
typedef struct moe_offload_rates {
    double expert_bytes;    /* weight bytes of one expert (3 * H * F * dtype size for SwiGLU) */
    double flops_per_pair;  /* FLOPs of one routed pair through one expert (6 * H * F) */
    double link_GBps;       /* host -> device copy rate */
    double host_GBps;       /* host FFN rate on expert weights (memory-bound regime) */
    double host_GFLOPs;     /* host FFN rate in FLOPs (compute-bound regime) */
    double gpu_GBps;        /* device FFN rate on expert weights */
} moe_offload_rates;

/*
 * Per-expert choice between the two execution paths of an offloaded expert
 * (Section IV-D.1): copy it to the GPU, or run it on the host where its weights
 * are.  For every expert that is not resident and has routed pairs:
 *   t_host = max(expert_bytes / host rate, counts[e] * flops_per_pair / host FLOP rate)
 *   t_gpu  = expert_bytes / link rate + expert_bytes / device rate
 * and an expert is a candidate for the copy when t_gpu < t_host -- few tokens
 * favour the host, many favour the copy.  Candidates are taken largest saving
 * first, at most max_copies, while taking one more still shortens the longer of
 * the two queues: the host's (the t_host of the experts it keeps, run one after
 * another on all its threads) and the link's (the t_gpu of the copied ones).
 *   counts [E], expert_slot [E] (host copies); choice [E] (host) out:
 *   1 = copy to the GPU, 0 = run on the host, -1 = resident or idle.
 * Host memory only; no device work.
 */
moe_status moe_offload_plan(int32_t experts, const int32_t* counts, const int32_t* expert_slot, int32_t slots,
                            const moe_offload_rates* rates, int32_t max_copies, int32_t* choice);

/*
 * Stage-boundary detection (Section IV-B.1, sliding-window pattern matching):
 * a finite-state machine over generated token ids recognises transition cues
 * (each a sequence of one or more token ids: a cue word split into subword
 * tokens) in every sequence of a batch, fed one token per sequence per decode
 * step.  Partial matches carry across steps, so a multi-token cue is reported
 * the step its last token arrives.  A match in any sequence is a stage
 * transition for the batch (Section IV-B.2 aggregates over all queries).
 * Host memory only; no device work.
 *
 * moe_cue_fsm_words: int32 words the machine needs for cues of `total_tokens`
 * tokens in all (5 * total_tokens + 8); -1 if total_tokens < 0.
 *
 * moe_cue_build: builds the machine into fsm [fsm_words] (caller-owned).
 *   cue_offsets [n_cues + 1]: cue c is cue_tokens[cue_offsets[c] .. cue_offsets[c+1]);
 *   cue_offsets[0] = 0, every cue has at least one token, token ids >= 0.
 *   n_cues = 0 builds a machine that never matches (offsets and tokens may be NULL).
 *   Identical cues are allowed; a match reports the lowest of their ids.
 *   Errors: MOE_ERR_INVALID_ARG for malformed cues, MOE_ERR_WORKSPACE if
 *   fsm_words < moe_cue_fsm_words(total); nothing is written then.
 *
 * moe_cue_step: advances `batch` sequences by one token each.
 *   tokens [batch]: the token each sequence generated this step; a negative id
 *   means none (the sequence is idle or finished): its window restarts.
 *   state [batch] in/out: 0 for a fresh sequence, else the value the previous
 *   call left.  matched [batch] out: id of the longest cue that ends with this
 *   token, or -1.  MOE_ERR_INVALID_ARG (nothing written) for a machine not made by
 *   moe_cue_build or a state out of range.
 */
int64_t moe_cue_fsm_words(int64_t total_tokens);
moe_status moe_cue_build(int32_t n_cues, const int32_t* cue_offsets, const int32_t* cue_tokens, int32_t* fsm,
                         int64_t fsm_words);
moe_status moe_cue_step(const int32_t* fsm, int32_t batch, const int32_t* tokens, int32_t* state,
                        int32_t* matched);

/*
 * Measurement utility (not a step of the method): reads `bytes` of device
 * memory at src once, with 16-byte loads spread over the whole GPU, so that the
 * caller can time the streaming-read rate of this GPU's HBM on its stream and
 * compare the weight-streaming FFN against it.
 *   src: device, 16-byte aligned; bytes >= 0, a multiple of 16.
 *   sink: device, one uint32 that is left unchanged in practice (a store
 *   conditioned on the data keeps the loads from being removed).
 */
moe_status moe_read_probe(const void* src, int64_t bytes, uint32_t* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SAEM_MOE_H */
