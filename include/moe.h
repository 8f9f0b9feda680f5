/*
 * moe.h -- C ABI of the MI355X (gfx950) Mixture-of-Experts FFN layer library
 * (libmoe.so).
 *
 * The layer is the sparse MoE FFN of Mixtral-8x7B, the model the paper's
 * serving engine is optimised for (Sec. 4.1, "Optimize Inference Engine";
 * Sec. 5, experimental settings).  Per token x (d values):
 *
 *   logits  l_e = sum_i x_i Wr[e,i] (+ b_e)                   router GEMM
 *   S       = the k largest logits; equal logits rank the lower expert first
 *   g_j     = softmax over the k selected logits (slot 0 = largest)
 *   FFN_e(x)= W2[e] (silu(W1[e] x) * (W3[e] x)),  silu(z) = z/(1+exp(-z))
 *   out     = sum_{j<k} g_j FFN_{S_j}(x)
 *
 * The engine batches requests continuously (Sec. 4.1, "Continuous Batching and
 * Batch Scheduler"), so T -- the tokens in this engine step, one per decoding
 * request or a prefill chunk -- changes on every call.  Every entry point takes
 * T at run time; nothing is recompiled and no call waits on the device.
 *
 * Conventions shared by every entry point:
 *   - Tensors are caller-owned DEVICE pointers, row-major, reduction index
 *     contiguous (the nn.Linear layout of Mixtral checkpoints):
 *       x [T,d] bf16, router_w [E,d] bf16, router_bias [E] f32,
 *       w1, w3 [E,ffn,d] bf16, w2 [E,d,ffn] bf16.
 *     The library keeps no reference after the call returns.
 *   - bf16 is passed as raw bits (moe_bf16_t).  Arithmetic: bf16 operands,
 *     f32 accumulation; logits, gate weights and slot outputs are f32; the
 *     SwiGLU intermediate h and the layer output are rounded to bf16 (RNE).
 *   - Calls are asynchronous and ordered on `stream` (NULL = the null
 *     stream).  Buffers must stay valid until that work has run.
 *   - Assignment a = t*k + j is slot j of token t.  Rows of the permuted
 *     (expert-major) order are r = 0..T*k-1; expert e owns rows
 *     [expert_offsets[e], expert_offsets[e+1]), in ascending a.
 *   - Limits: 1 <= E <= 64, 1 <= k <= min(E, 8), d and ffn multiples of 64
 *     with d <= 65536 and ffn <= 65536, 0 <= T and T*k < 2^31.  Device
 *     pointers must be 16-byte aligned.  T = 0 returns MOE_OK and launches
 *     nothing; buffers whose size scales with T may then be NULL.
 *   - Errors: every argument is checked before anything is enqueued; on
 *     error nothing is enqueued and a message is available from
 *     moe_last_error() (thread-local).  A failed launch returns MOE_ERR_HIP.
 *     Faults inside kernels surface at the caller's next synchronisation.
 *     No C++ exception crosses this interface.
 */
#ifndef MOE_MI355X_H
#define MOE_MI355X_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t moe_bf16_t; /* raw bfloat16 bits */

typedef enum {
    MOE_OK = 0,
    MOE_ERR_INVALID_ARG = 1, /* null/misaligned pointer, bad size, aliasing */
    MOE_ERR_UNSUPPORTED = 2, /* outside the limits above */
    MOE_ERR_NO_MEMORY = 3,   /* workspace too small or allocation failed */
    MOE_ERR_HIP = 4          /* a HIP runtime call or kernel launch failed */
} moe_status_t;

/*
 * Router GEMM + top-k gating + dispatch (Sec. 4.1: the MoE router of the
 * Mixtral model the engine serves).
 *   logits[t,e]   = sum_i x[t,i] router_w[e,i] in f32 (+ router_bias[e], f32,
 *                   added after the sum; NULL = no bias).  Never rounded to bf16.
 *   topk_ids[t,j] = j-th ranked expert of token t (larger logit first; equal
 *                   logits: lower index first).                         [T,k] i32
 *   topk_w[t,j]   = exp(l_{S_j} - l_{S_0}) / sum_m exp(l_{S_m} - l_{S_0}) [T,k] f32
 *   expert_offsets[e] = number of assignments to experts < e; [E] = T*k. [E+1] i32
 *   perm[r]       = assignment a of permuted row r (expert-major, then a). [T*k] i32
 *   logits        = optional [T,E] f32 copy of the router logits (NULL to skip).
 */
moe_status_t moe_route(const moe_bf16_t* x, const moe_bf16_t* router_w, const float* router_bias,
                       int64_t T, int32_t d, int32_t E, int32_t k, int32_t* topk_ids,
                       float* topk_w, int32_t* expert_offsets, int32_t* perm, float* logits,
                       hipStream_t stream);

/*
 * Token-to-expert permutation (Sec. 4.1, MoE layer): gather token rows into
 * per-expert contiguous rows.  x_perm[r,:] = x[perm[r] / k, :].  [T*k,d] bf16.
 * x_perm must not overlap x.
 */
moe_status_t moe_permute(const moe_bf16_t* x, const int32_t* perm, int64_t T, int32_t d,
                         int32_t k, moe_bf16_t* x_perm, hipStream_t stream);

/*
 * Expert stages (moe_swiglu_up/down, their _fp8 forms, moe_grouped_swiglu):
 * E is the number of experts whose weights are passed.  It may be a shard of
 * the routed experts (expert parallelism: pass the shard's weights and its
 * slice of the offsets, whose row numbers stay absolute), so k may exceed it
 * here; 1 <= k <= 8 still holds.
 *
 * First half of the per-expert SwiGLU FFN (Sec. 4.1, Mixtral experts):
 * for every expert e and row r in [expert_offsets[e], expert_offsets[e+1]):
 *   h[r,n] = bf16( silu(sum_i w1[e,n,i] xr[i]) * sum_i w3[e,n,i] xr[i] )
 * where the token row xr is x[perm[r] / k, :] when perm is given (the gather
 * of moe_permute fused into the GEMM; x is then [T,d]) and x[r, :] when perm
 * is NULL (x is then the permuted [T*k,d] rows).  h [T*k,ffn] bf16.
 */
moe_status_t moe_swiglu_up(const moe_bf16_t* x, const int32_t* perm,
                           const int32_t* expert_offsets, const moe_bf16_t* w1,
                           const moe_bf16_t* w3, int64_t T, int32_t d, int32_t ffn, int32_t E,
                           int32_t k, moe_bf16_t* h, hipStream_t stream);

/*
 * Second half of the expert FFN with the gate-weighted scatter fused in
 * (Sec. 4.1, the Mixtral experts of the served model: the W2 projection of
 * each SwiGLU expert, then the gate-weighted sum of the k expert outputs):
 * for every expert e and row r of e, with a = perm[r]:
 *   y[a,i] = topk_w[a] * sum_n w2[e,i,n] h[r,n]        (f32, assignment order)
 * If topk_w or perm is NULL the plain result is written in row order instead:
 *   y[r,i] = sum_n w2[e,i,n] h[r,n].
 * h [T*k,ffn] bf16, y [T*k,d] f32.
 */
moe_status_t moe_swiglu_down(const moe_bf16_t* h, const int32_t* expert_offsets,
                             const moe_bf16_t* w2, const float* topk_w, const int32_t* perm,
                             int64_t T, int32_t d, int32_t ffn, int32_t E, int32_t k, float* y,
                             hipStream_t stream);

/*
 * The W2 projection of the experts (Sec. 4.1, Mixtral's SwiGLU experts, as
 * in moe_swiglu_down) with its reduction over ffn cut into parts (the same sums:
 * y of moe_swiglu_down = the sum of the slices written here), for prefill
 * sizes where the persistent tiled kernel runs (more than 64 rows per
 * expert on average) and a few hundred output tiles would leave its last
 * round of workgroups mostly idle.  y is [max_parts, T*k, d] f32: slice s
 * receives the partial sum over the s-th part of ffn, gate-weighted and
 * scattered as in moe_swiglu_down.  The number of parts used (a power of two
 * up to 16, at most max_parts, each part at least 512 elements of ffn) is
 * chosen on the device from the routed row counts and stored to *parts
 * (device int32, 4-byte aligned).  Where max_parts >= 4 and slices 1 ..
 * max_parts-1 together hold at least 256 x 65536 floats plus a 4 KiB table
 * (prefill sizes), the tiles are instead left uncut and only the tiles of
 * the persistent grid's last, partial round are split across its idle
 * workgroups; those pieces go to slices 1.. as scratch and a second kernel
 * adds them into slice 0 (in piece order), so *parts = 1 on return and the
 * rest of slices 1.. holds scratch.  In the streaming regime (up to 64 rows per
 * expert on average) with T > 64, the experts holding more than 64 rows take
 * the cut tiled kernel and their slices are then added into slice 0 in
 * ascending order, so *parts = 1 on return; the other experts stream uncut
 * into slice 0.  Where only the streaming kernel runs, *parts = 1.  Except
 * with the tail split, slices at or past the count used are left as they
 * were.  moe_combine_parts sums the
 * slices; moe_forward runs this pair.  Errors as moe_swiglu_down, and
 * MOE_ERR_INVALID_ARG for max_parts < 1 or parts NULL.
 */
moe_status_t moe_swiglu_down_parts(const moe_bf16_t* h, const int32_t* expert_offsets,
                                   const moe_bf16_t* w2, const float* topk_w, const int32_t* perm,
                                   int64_t T, int32_t d, int32_t ffn, int32_t E, int32_t k,
                                   int32_t max_parts, float* y, int32_t* parts,
                                   hipStream_t stream);

/*
 * The grouped SwiGLU expert FFN on permuted rows (Sec. 4.1, the experts of
 * the Mixtral MoE layer the engine serves; Sec. 5, Mixtral-8x7B):
 * moe_swiglu_up(x_perm, perm = NULL) into h_ws, then moe_swiglu_down into y
 * (same meaning of topk_w / perm as there).
 * h_ws is caller scratch of T*k*ffn bf16.
 */
moe_status_t moe_grouped_swiglu(const moe_bf16_t* x_perm, const int32_t* expert_offsets,
                                const moe_bf16_t* w1, const moe_bf16_t* w3,
                                const moe_bf16_t* w2, const float* topk_w, const int32_t* perm,
                                int64_t T, int32_t d, int32_t ffn, int32_t E, int32_t k,
                                moe_bf16_t* h_ws, float* y, hipStream_t stream);

/*
 * Gate-weighted un-permute/combine (Sec. 4.1, the Mixtral MoE layer: a
 * token's output is the gate-weighted sum of its k experts' outputs; the
 * residual add is the pre-norm block around the layer): slots of a token are
 * summed in ascending j in f32, after the optional residual:
 *   s = (residual ? residual[t,i] : 0) + y[t*k+0,i] + ... + y[t*k+k-1,i]
 *   out[t,i] = bf16(s) (if out), out_f32[t,i] = s (if out_f32).
 * y [T*k,d] f32 in assignment order (already gate-weighted), residual/out_f32
 * [T,d] f32, out [T,d] bf16.  At least one of out/out_f32.  out_f32 may equal
 * residual (in-place residual update); nothing else may overlap.
 */
moe_status_t moe_combine(const float* y, const float* residual, int64_t T, int32_t d, int32_t k,
                         moe_bf16_t* out, float* out_f32, hipStream_t stream);

/*
 * The gate-weighted combine (Sec. 4.1, as in moe_combine) over the slices of
 * moe_swiglu_down_parts: y [max_parts,T*k,d]
 * f32; each slot first sums its slices 0 .. n-1 in ascending order, with n =
 * *parts (device int32, read by the kernel, clamped to [1, max_parts]), then
 * the slots are summed as in moe_combine.
 */
moe_status_t moe_combine_parts(const float* y, const int32_t* parts, int32_t max_parts,
                               const float* residual, int64_t T, int32_t d, int32_t k,
                               moe_bf16_t* out, float* out_f32, hipStream_t stream);

/*
 * The whole MoE FFN layer of the served model (Sec. 4.1, "Optimize Inference
 * Engine": the engine work targets Mixture-of-Experts models; Sec. 5:
 * Mixtral-8x7B, up to 256 concurrent requests per step under continuous
 * batching): route -> SwiGLU experts (the gather of token rows is fused
 * into the first expert GEMM) -> combine.  Where both expert GEMMs run on the
 * weight-streaming kernels with at most 1024 assignments (decode steps), the
 * expert offsets and row order are built from the top-k ids inside those
 * kernels and no separate dispatch runs; the results are bitwise those of the
 * stage-by-stage calls.  out [T,d] bf16, must not overlap
 * any input.  Scratch is owned by the library, cached per device and grown on
 * demand (a growth is refused with MOE_ERR_NO_MEMORY while `stream` is being
 * captured into a graph; call once outside capture first).  A buffer that was
 * handed to a call under capture is kept alive when a later call grows the
 * scratch, so graphs captured earlier stay valid (until
 * moe_release_workspace).  The environment variable MOE_WORKSPACE_LIMIT_BYTES
 * (a decimal byte count, read on every call) caps each library-owned scratch
 * buffer: a call that needs more returns MOE_ERR_NO_MEMORY before any HIP
 * call (an unparsable value gives MOE_ERR_INVALID_ARG).  Every call on one
 * device shares that scratch, so calls on different streams of one device
 * must not overlap in time; give each stream its own caller workspace
 * (moe_forward_ex) to run them concurrently.
 * At prefill sizes (up to 4 parts) and for the heavy experts of a streaming
 * step with T > 64 (up to 2 parts) the down GEMM runs as
 * moe_swiglu_down_parts and the combine as moe_combine_parts (the part count
 * depends on the routed row counts and the GPU's compute units), so the
 * result can differ in the last bits from the uncut staged calls
 * moe_grouped_swiglu + moe_combine; for the same inputs on the same GPU it is
 * deterministic.
 */
moe_status_t moe_forward(const moe_bf16_t* x, const moe_bf16_t* router_w, const moe_bf16_t* w1,
                         const moe_bf16_t* w3, const moe_bf16_t* w2, int64_t T, int32_t d,
                         int32_t ffn, int32_t E, int32_t k, moe_bf16_t* out, hipStream_t stream);

/*
 * moe_forward with the options of a residual block (Sec. 4.1 and Sec. 5: the
 * MoE layer inside Mixtral's pre-norm decoder layer, whose residual stream
 * the caller keeps in f32):
 *   router_bias  [E] f32 or NULL;
 *   residual     [T,d] f32 or NULL, added before rounding (see moe_combine);
 *   out          [T,d] bf16 or NULL; out_f32 [T,d] f32 or NULL (at least one;
 *                out_f32 may equal residual);
 *   workspace    caller device scratch of at least
 *                moe_workspace_size(T,d,ffn,E,k) bytes, 256-byte aligned, or
 *                NULL for the library-owned scratch.
 */
moe_status_t moe_forward_ex(const moe_bf16_t* x, const moe_bf16_t* router_w,
                            const float* router_bias, const moe_bf16_t* w1,
                            const moe_bf16_t* w3, const moe_bf16_t* w2, int64_t T, int32_t d,
                            int32_t ffn, int32_t E, int32_t k, const float* residual,
                            moe_bf16_t* out, float* out_f32, void* workspace,
                            size_t workspace_bytes, hipStream_t stream);

/*
 * moe_forward_ex without a workspace, for callers that cannot allocate device
 * memory: code under graph capture, tight serving loops, harnesses that
 * forbid allocation.  The call allocates nothing (no hipMalloc, no stream or
 * event creation: the heavy and light expert launches of a split step run in
 * sequence on `stream`).  Its scratch is one fixed 64 MiB device array in the
 * library, one copy per GPU, held from the library's load until the process
 * ends; sizes whose moe_workspace_size exceeds 64 MiB (e.g. Mixtral shapes
 * above about 512 tokens) return MOE_ERR_NO_MEMORY before anything is
 * enqueued.  Every call on one GPU shares that GPU's array, which keeps the
 * last call's contents: calls that overlap in time on one GPU (on different
 * streams or host threads) race, and must be ordered by the caller.  Nothing
 * in the array needs clearing between calls.  Arguments and results as
 * moe_forward_ex (workspace omitted).
 */
moe_status_t moe_forward_noalloc(const moe_bf16_t* x, const moe_bf16_t* router_w,
                                 const float* router_bias, const moe_bf16_t* w1,
                                 const moe_bf16_t* w3, const moe_bf16_t* w2, int64_t T, int32_t d,
                                 int32_t ffn, int32_t E, int32_t k, const float* residual,
                                 moe_bf16_t* out, float* out_f32, hipStream_t stream);

/*
 * 8-bit expert weights (Sec. 4.1, "Model Quantization": weights stored as
 * 8-bit floats; Sec. 5 serves an 8-bit quantized Mixtral-8x7B).  Each expert
 * matrix is held as OCP FP8 E4M3 bytes -- sign, 4 exponent bits with bias 7,
 * 3 mantissa bits; exponent 0 is subnormal (m/8 * 2^-6); S.1111.111 is NaN;
 * largest finite value 448 -- with one f32 scale per weight row:
 *   w1[e,n,i] = e4m3(w1q[e,n,i]) * w1s[e,n]     w1q, w3q [E,ffn,d] u8, w1s, w3s [E,ffn] f32
 *   w2[e,i,n] = e4m3(w2q[e,i,n]) * w2s[e,i]     w2q [E,d,ffn] u8,  w2s [E,d] f32
 * The E4M3 values convert exactly to bf16 operands, products accumulate in
 * f32 and each row's sum is multiplied by its scale; everything else (token
 * rows, h, y, out, routing) is as in the bf16 calls of the same name, with
 * the same limits and alignment rules (byte arrays and scales 16-byte
 * aligned).  A NaN byte, or a non-finite scale, makes the rows it reaches
 * NaN.  Kernel families as for bf16 weights (moe_set_gemm_variant): the
 * tiled kernels stage the E4M3 bytes in LDS and widen them to bf16 operands
 * there.
 */
moe_status_t moe_swiglu_up_fp8(const moe_bf16_t* x, const int32_t* perm,
                               const int32_t* expert_offsets, const uint8_t* w1q,
                               const float* w1s, const uint8_t* w3q, const float* w3s, int64_t T,
                               int32_t d, int32_t ffn, int32_t E, int32_t k, moe_bf16_t* h,
                               hipStream_t stream);

moe_status_t moe_swiglu_down_fp8(const moe_bf16_t* h, const int32_t* expert_offsets,
                                 const uint8_t* w2q, const float* w2s, const float* topk_w,
                                 const int32_t* perm, int64_t T, int32_t d, int32_t ffn, int32_t E,
                                 int32_t k, float* y, hipStream_t stream);

/* moe_swiglu_down_parts with the 8-bit weights above (same slices, count and
 * errors). */
moe_status_t moe_swiglu_down_parts_fp8(const moe_bf16_t* h, const int32_t* expert_offsets,
                                       const uint8_t* w2q, const float* w2s, const float* topk_w,
                                       const int32_t* perm, int64_t T, int32_t d, int32_t ffn,
                                       int32_t E, int32_t k, int32_t max_parts, float* y,
                                       int32_t* parts, hipStream_t stream);

/* moe_forward_ex with the 8-bit expert weights above (the router stays bf16). */
moe_status_t moe_forward_fp8_ex(const moe_bf16_t* x, const moe_bf16_t* router_w,
                                const float* router_bias, const uint8_t* w1q, const float* w1s,
                                const uint8_t* w3q, const float* w3s, const uint8_t* w2q,
                                const float* w2s, int64_t T, int32_t d, int32_t ffn, int32_t E,
                                int32_t k, const float* residual, moe_bf16_t* out,
                                float* out_f32, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/*
 * RMSNorm of the f32 residual stream, as in front of each MoE block of a
 * pre-norm residual stack (Mixtral's layer structure, Sec. 4.1 citation):
 *   a[t,i] = bf16( h[t,i] / sqrt(mean_i h[t,i]^2 + eps) * gamma[i] )
 * h [T,d] f32, gamma [d] bf16, a [T,d] bf16, eps >= 0.
 */
moe_status_t moe_rmsnorm(const float* h, const moe_bf16_t* gamma, int64_t T, int32_t d, float eps,
                         moe_bf16_t* a, hipStream_t stream);

/*
 * ---- The decoder layer around the MoE block (one decode step) -------------
 * The engine serves the whole model with paged, flash-style attention (Sec. 2;
 * Sec. 4.1, "Other Optimizations").  With the calls below and moe_rmsnorm,
 * moe_combine and moe_forward_ex, one decoder layer of a decode step runs on
 * the device for T tokens, one per request:
 *   a = RMSNorm(h) gamma_attn (bf16)        moe_rmsnorm
 *   qkv = a [Wq; Wk; Wv]^T (f32)            moe_linear
 *   RoPE(q, k); k, v -> cache (bf16)        moe_rope_kv_append
 *   o = attention over the cache (bf16)     moe_attention_decode
 *   h += o Wo^T (f32 residual)              moe_linear + moe_combine (k = 1)
 *   h += MoE(RMSNorm(h) gamma_moe)          moe_rmsnorm + moe_forward_ex
 * KV cache layout, keys and values alike: [npages, Hkv, page, hd] bf16; the
 * request of token t stores position s in page page_table[t * maxp + s /
 * page], slot s % page.  Page ids, positions and context lengths are device
 * data: the kernels clamp values outside the cache (invalid input) so that
 * nothing outside the cache is read or written.
 */

/*
 * Dense projection y[t, n] = sum_i x[t, i] w[n, i] (bf16 operands, f32
 * accumulate and output): x [T, K] bf16, w [N, K] bf16 (nn.Linear layout),
 * y [T, N] f32.  K, N multiples of 64 (<= 65536).  The weight-streaming GEMM
 * with one matrix, or, from 128 output tiles of 256 x 256 on (N a multiple of
 * 256, K of 128; e.g. N = 6144 from 1281 tokens), the tiled MFMA GEMM.
 */
moe_status_t moe_linear(const moe_bf16_t* x, const moe_bf16_t* w, int64_t T, int32_t K, int32_t N,
                        float* y, hipStream_t stream);

/*
 * Rotary position embedding and KV-cache append for the new token of each
 * request.  qkv [T, (Hq + 2 Hkv) hd] f32 holds the token's query heads, then
 * key heads, then value heads; pos [T] its position (the number of positions
 * already cached).  Query and key heads are rotated, element i with element
 * i + hd/2, by the angle pos * theta^(-2i/hd) (the rotate-half layout of
 * Mixtral/Llama checkpoints; Mixtral: theta = 1e6).  Writes q_out [T, Hq, hd]
 * and the key and value rows at position pos[t], all rounded to bf16.  hd even.
 */
moe_status_t moe_rope_kv_append(const float* qkv, const int32_t* pos, const int32_t* page_table,
                                int64_t T, int32_t Hq, int32_t Hkv, int32_t hd, int32_t page,
                                int32_t maxp, int64_t npages, double theta, moe_bf16_t* q_out,
                                moe_bf16_t* k_cache, moe_bf16_t* v_cache, hipStream_t stream);

/*
 * Grouped-query decode attention over the paged cache (PagedAttention, with
 * FlashAttention's one-pass softmax):
 *   out[t, h, :] = sum_{s < ctx[t]} softmax_s(scale q[t,h,:] . K_s) V_s
 * with K_s, V_s of KV head h / (Hq / Hkv) of token t's request.  q [T, Hq, hd]
 * bf16, out [T, Hq * hd] bf16 (f32 softmax and accumulation).  ctx[t] in
 * [1, maxp * page].  Supported: hd = 128, Hq / Hkv in {1, 2, 4, 8}, page a
 * multiple of 8, maxp <= 4096 (MOE_ERR_UNSUPPORTED otherwise).  When T * Hkv
 * is small and contexts long, the positions are split over several
 * workgroups whose partial states go to library-owned scratch (per device,
 * grown on demand like moe_forward's, refused with MOE_ERR_NO_MEMORY while
 * `stream` is captured into a graph if it must grow) and are merged in a
 * fixed order: results do not depend on the split.  Calls that use this
 * scratch on one device must not overlap on different streams.
 */
moe_status_t moe_attention_decode(const moe_bf16_t* q, const moe_bf16_t* k_cache,
                                  const moe_bf16_t* v_cache, const int32_t* page_table,
                                  const int32_t* ctx, int64_t T, int32_t Hq, int32_t Hkv,
                                  int32_t hd, int32_t page, int32_t maxp, int64_t npages,
                                  float scale, moe_bf16_t* out, hipStream_t stream);

/*
 * Frees the library-owned scratch of the current device (moe_forward's and
 * moe_attention_decode's, and buffers kept alive for captured graphs) after
 * waiting for all work on the device.  Graphs captured earlier whose calls
 * used the library scratch must not be replayed afterwards; the next call
 * allocates again.  Not while a stream of the device is being captured.
 */
moe_status_t moe_release_workspace(void);

/* Bytes of scratch moe_forward_ex needs for these sizes (0 for invalid sizes). */
size_t moe_workspace_size(int64_t T, int32_t d, int32_t ffn, int32_t E, int32_t k);

/*
 * Expert-GEMM kernel family used by moe_swiglu_up/down and the forward calls:
 *   0 = automatic, 1 = weight-streaming (decode shapes), 2 = tiled (prefill
 *   shapes).  Automatic: streaming while T*k/E <= 64, tiled above; in the
 *   streaming regime with T > 64 (so an expert may hold more than 64 rows)
 *   each expert GEMM is two launches that split the experts on the device by
 *   their row count (<= 64: streaming; more: tiled for the up GEMM, and for
 *   the down GEMM where the caller provides reduction-part slices, streaming
 *   with 128-row passes otherwise).  Process-wide; returns the previous
 *   value, or -1 for an unknown value (nothing changed).  For testing and
 *   measurement.  The same choice applies to the 8-bit weight calls.
 */
int moe_set_gemm_variant(int variant);

/* The kernel family the expert GEMMs use for these sizes under the
 * current moe_set_gemm_variant setting: 1 = weight-streaming, 2 = tiled,
 * 3 = split by rows per expert (see moe_set_gemm_variant); 0 for invalid
 * sizes.  Host-only, enqueues nothing. */
int moe_gemm_variant_for(int64_t T, int32_t d, int32_t ffn, int32_t E, int32_t k);

/* Static text of a status code. */
const char* moe_status_string(int status);

/* Message of the last error on the calling thread ("" if none). */
const char* moe_last_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int moe_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MOE_MI355X_H */
