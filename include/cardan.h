/*
 * cardan.h -- C ABI of libcardan.so, an MI355X (gfx950) implementation of one
 * batch-1-to-64 Mixture-of-Experts decode layer whose expert matrices are
 * stored compressed.
 *
 * The layer (paper Sec. 2.1): a router scores the E experts for every token,
 * keeps the top-k and weights them with a softmax over the k kept logits;
 * every kept expert runs gate and up projections, the SiLU-gated product
 * p = silu(g) * u, and a down projection; the layer output is the
 * affinity-weighted sum of the expert outputs.
 *
 * Expert representation (paper Sec. 2.3 and Sec. 3.1, Eq. (1)): a gate or up
 * matrix W_e [H, I] is Q_B(J_e) + U V_e, where Q_B(J_e) is rebuilt from a
 * shared code book B [K, d] and a private uint8 index map J_e [H/d, I] (block
 * b of column j is code word J_e[b, j], whose element i sits at input row
 * b*d + i), U [H, r] is a basis shared by all experts and V_e [r, I] holds
 * private coefficients. The down matrix [I, H] is Q_B(J^d_e) + A_e B with
 * private A_e [I, r] and a shared output-side basis B [r, H].
 *
 * Conventions for every entry point:
 *   - bf16 values are raw bit patterns (uint16_t); all arrays are dense and
 *     row-major in the shapes given; every pointer is a DEVICE pointer,
 *     16-byte aligned, owned by the caller and only read during the call
 *     (outputs are written). The library never allocates, frees or
 *     synchronises inside these calls and keeps no pointer after returning.
 *   - All work is enqueued on `stream` and the call returns without waiting.
 *     Buffers must stay valid until the stream has passed the work.
 *   - Arguments are validated before anything is enqueued; on any error
 *     nothing is launched, a negative code is returned and
 *     cardan_last_error() describes it.
 *   - `ws` is a caller-owned device workspace of at least
 *     cardan_workspace_bytes() bytes. It must be zero-filled once before its
 *     first use; every completed call leaves it ready for the next. Calls
 *     that overlap in time must not share a workspace.
 *   - Supported shapes: d in {2, 4, 8}; 1 <= K <= 256; H % 64 == 0;
 *     I % 32 == 0; 1 <= E <= 1024; 1 <= top_k <= min(E, 32); 0 <= r <= 512;
 *     1 <= B <= 64. Other shapes return CARDAN_ERR_UNSUPPORTED or
 *     CARDAN_ERR_BAD_SHAPE.
 *   - Code values >= K read zero code words (memory-safe); expert indices
 *     outside [0, E) passed to cardan_vq_lr_expert_ffn contribute nothing.
 *   - The first int32 of the workspace (CARDAN_WS_STATUS_OFFSET) counts
 *     internal waits that gave up after their bound (seconds); nonzero means
 *     the results of the calls since it was last zero are invalid. The
 *     library never clears it; the caller may.
 *   - The layer kernels are persistent: each launches at most as many
 *     workgroups as the device holds at once and their work items wait on
 *     one another. They need the device's compute units to themselves while
 *     they run; other resident work (another stream or process) can keep
 *     workgroups from starting, and the waits that depend on them then give
 *     up into the status count above (the results are invalid, nothing hangs).
 *   - A workspace serves one (H, I, E): its counter offsets depend on those
 *     three only, so calls of any batch, rank, block length or expert-weight
 *     form on that shape may share it in turn; zero it again before using it
 *     for another (H, I, E).
 *   - Reentrancy: the entry points keep no mutable host state apart from the
 *     thread-local error text and an occupancy cache guarded by a mutex; host
 *     threads may call them concurrently on separate workspaces. The
 *     profiling hooks below are the exception (host-global, not thread-safe).
 */
#ifndef CARDAN_H
#define CARDAN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Same declaration as HIP's own; lets this header stand alone. */
typedef struct ihipStream_t* hipStream_t;
typedef struct ihipEvent_t* hipEvent_t;

#define CARDAN_ABI_VERSION 1
#define CARDAN_WS_STATUS_OFFSET 0

enum {
  CARDAN_OK = 0,
  CARDAN_ERR_NULL_PTR = -1,   /* a required pointer is NULL               */
  CARDAN_ERR_BAD_SHAPE = -2,  /* shape or batch outside the valid domain  */
  CARDAN_ERR_UNSUPPORTED = -3,/* valid but not compiled (e.g. d == 16)    */
  CARDAN_ERR_WORKSPACE = -4,  /* ws_bytes below cardan_workspace_bytes()  */
  CARDAN_ERR_HIP = -5,        /* a HIP launch or event call failed        */
  CARDAN_ERR_ALIGN = -6       /* a pointer is not 16-byte aligned         */
};

typedef uint16_t cardan_bf16;

/* Layer shape: hidden size H, expert intermediate size I, E experts, top_k
 * selected per token, VQ block length d, K code words, rank r (Table 1). */
typedef struct {
  int32_t H, I, E, top_k, d, K, r;
} cardan_shape;

/* One layer's weights (device pointers). With r == 0 the six low-rank
 * pointers may be NULL. U_up may equal U_gate (one basis for both). */
typedef struct {
  const cardan_bf16* router_w;    /* [H][E]                                  */
  const float*       router_bias; /* [E] added to the logits, or NULL        */
  const cardan_bf16* cb_gate;     /* [K][d] shared gate code book            */
  const cardan_bf16* cb_up;       /* [K][d] shared up code book              */
  const cardan_bf16* cb_down;     /* [K][d] shared down code book            */
  const uint8_t*     codes_gate;  /* [E][H/d][I] private index maps          */
  const uint8_t*     codes_up;    /* [E][H/d][I]                             */
  const uint8_t*     codes_down;  /* [E][I/d][H]                             */
  const cardan_bf16* U_gate;      /* [H][r] shared basis (gate)              */
  const cardan_bf16* U_up;        /* [H][r] shared basis (up)                */
  const cardan_bf16* V_gate;      /* [E][r][I] private coefficients          */
  const cardan_bf16* V_up;        /* [E][r][I]                               */
  const cardan_bf16* A_down;      /* [E][I][r] private down factor           */
  const cardan_bf16* B_down;      /* [r][H] shared output-side down basis    */
} cardan_layer;

/* ABI version of the loaded library (CARDAN_ABI_VERSION). */
int cardan_abi_version(void);

/* Text of the last error on the calling thread ("" if none). Valid until the
 * next cardan_* call on the same thread. */
const char* cardan_last_error(void);

/* Workspace size in bytes needed by every ws-taking entry point for this
 * shape and any batch up to B (the dense-weight entry points and the decode
 * step included).
 * Host-only; no device is touched. */
int cardan_workspace_bytes(const cardan_shape* shape, int32_t B, size_t* out);

/* Router and gating (paper Sec. 2.1): logits l[t][e] = sum_h x[t][h] *
 * router_w[h][e] + router_bias[e], accumulated in float64 from the exact bf16
 * products; the top_k experts by descending logit (exact ties to the lower
 * index) go to topk_idx[B][top_k] (int32, in that order) and their softmax
 * over the top_k logits to topk_w[B][top_k] (float32).
 * x: [B][H] bf16. */
int cardan_route_topk(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                      const cardan_bf16* router_w, const float* router_bias,
                      int32_t* topk_idx, float* topk_w,
                      void* ws, size_t ws_bytes, hipStream_t stream);

/* Shared projections of Eq. (1) (paper Sec. 4.2, computed once per token):
 * z[0][t][q] = sum_h U_gate[h][q] x[t][h] and z[1][t][q] likewise with U_up,
 * as float32 z[2][B][r]. Both halves are always written; U_up may equal
 * U_gate. Requires r > 0. */
int cardan_shared_proj(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                       const cardan_bf16* U_gate, const cardan_bf16* U_up, float* z,
                       void* ws, size_t ws_bytes, hipStream_t stream);

/* Expert computation and weighted combine for a given routing (Sec. 2.1,
 * Eq. (1)): tokens are grouped by expert so each selected expert's codes are
 * read once; for every (token, selected expert) g and u are the VQ gather sum
 * plus V^T z (one float32 accumulation), p = silu(g) * u, the down output is
 * Q^T p + B^T (A^T p), and y[t] = sum_j topk_w[t][j] * y_{topk_idx[t][j]}.
 * topk_idx/topk_w: [B][top_k] as produced by cardan_route_topk; z: [2][B][r]
 * as produced by cardan_shared_proj (may be NULL iff r == 0);
 * y: [B][H] float32 output. */
int cardan_vq_lr_expert_ffn(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                            const int32_t* topk_idx, const float* topk_w, const float* z,
                            const cardan_layer* layer, float* y,
                            void* ws, size_t ws_bytes, hipStream_t stream);

/* The whole layer (paper Sec. 2.1 with the experts of Sec. 3.1, Eq. (1), and
 * the once-per-token shared projections and cross-expert batching of
 * Sec. 4.2): route + top-k + gating as cardan_route_topk, z = U^T x as
 * cardan_shared_proj, then the grouped expert computation and weighted
 * combine of cardan_vq_lr_expert_ffn. Writes y [B][H] float32 and the
 * routing topk_idx [B][top_k] int32, topk_w [B][top_k] float32.
 * Gate/up form: the VQ part is decoded from code words on the matrix cores;
 * with the environment variable CARDAN_GATEUP=tbook (read at every call of
 * this entry point and of cardan_moe_layer_relu2) one-token experts sum the
 * per-token projection code book T[b][k] = x_b . cb_k of Sec. 4.2 instead
 * (d = 4 or 8, K a multiple of 4, at most 64 MiB of T; otherwise the code
 * words). Both give the same result up to float32 rounding. */
int cardan_moe_layer(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                     const cardan_layer* layer, float* y, int32_t* topk_idx, float* topk_w,
                     void* ws, size_t ws_bytes, hipStream_t stream);

/* The whole layer with up-only experts and a squared-ReLU activation (the
 * expert form of the paper's Nemotron-3 model, Table 2 "up" and the fidelity
 * test of Sec. 5.7): routing and z = U_up^T x as cardan_moe_layer, then for
 * every (token, selected expert) u = VQ gather sum + V_up^T z, p =
 * max(u, 0)^2, the down output Q^T p + B^T (A^T p), and the weighted combine.
 * The gate fields of `layer` (cb_gate, codes_gate, U_gate, V_gate) are not
 * read and may be NULL. Outputs, workspace and errors as cardan_moe_layer. */
int cardan_moe_layer_relu2(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                           const cardan_layer* layer, float* y, int32_t* topk_idx, float* topk_w,
                           void* ws, size_t ws_bytes, hipStream_t stream);

/* One decode step through n_layers stacked MoE layers (the 48-layer workload
 * of the paper's Qwen3 decoding, attention omitted): layer 0 reads x0
 * [B][H] bf16; layer l + 1 reads x_{l+1} = bf16_rne(y_l / sqrt(mean_h(y_l^2)
 * + eps)) of layer l's output y_l (no learned scale), as cardan_rmsnorm_bf16
 * would form it; y [B][H] float32 receives the last layer's output. Every
 * layer is cardan_moe_layer on its own weights layers[l] (Sec. 2.1, Sec. 3.1
 * Eq. (1), Sec. 4.2), all with the same shape. Per layer l the routing goes
 * to topk_idx / topk_w [n_layers][B][top_k]; x_norm, if not NULL, receives
 * the normalised inputs of layers 1..n_layers-1 as [n_layers - 1][B][H] bf16.
 * The normalisation runs inside the next layer's routing kernel (the layer's
 * combine writes per-token partial sums of y^2), so a layer costs two kernel
 * launches. With the environment variable CARDAN_PREFETCH set to "1" the
 * expert kernel's idle workgroups also read the next layer's router weights,
 * bases and code books ahead of its routing kernel (the paper's overlap of
 * routing-independent reads, Sec. 4.1); it changes no output and is off by
 * default because it measured slower. ws: at least
 * cardan_workspace_bytes(shape, B) bytes; one workspace serves every layer.
 * 1 <= n_layers <= 4096, eps finite and >= 0. */
int cardan_moe_decode_step(const cardan_shape* shape, int32_t B, int32_t n_layers, const cardan_bf16* x0,
                           const cardan_layer* layers, float eps, float* y, cardan_bf16* x_norm,
                           int32_t* topk_idx, float* topk_w, void* ws, size_t ws_bytes,
                           hipStream_t stream);

/* Size of the library's own scratch array, one per GPU (16 MiB). */
#define CARDAN_SCRATCH_BYTES (16u << 20)

/* cardan_moe_layer without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc. The kernels use a fixed device-resident
 * scratch array of CARDAN_SCRATCH_BYTES inside the library (each GPU the
 * library runs on holds its own copy until the process ends); this call
 * allocates nothing (no hipMalloc, hipFree or allocating library routine).
 * Arguments, outputs, results and errors are those of cardan_moe_layer; a
 * layer whose workspace at this batch exceeds the array returns
 * CARDAN_ERR_WORKSPACE before anything is enqueued.
 * Every call on a GPU shares that GPU's array, which keeps the last call's
 * contents: calls that overlap in time on one GPU (several streams or host
 * threads) race and give undefined results, so serialise them. A call whose
 * (H, I, E) differs from the previous call's on the GPU, the first call, and
 * any call recorded under graph capture enqueue a small zero-fill kernel of
 * the array's counters before the layer. The wait-timeout status count of
 * these calls is not readable (cardan_moe_layer with a workspace reports it). */
int cardan_moe_layer_noalloc(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                             const cardan_layer* layer, float* y, int32_t* topk_idx,
                             float* topk_w, hipStream_t stream);

/* Dense bf16 expert weights of an uncompressed layer (device pointers). */
typedef struct {
  const cardan_bf16* router_w;    /* [H][E]                                  */
  const float*       router_bias; /* [E] added to the logits, or NULL        */
  const cardan_bf16* W_gate;      /* [E][H][I]                               */
  const cardan_bf16* W_up;        /* [E][H][I]                               */
  const cardan_bf16* W_down;      /* [E][I][H]                               */
} cardan_dense_layer;

/* The layer with compressed gate and up projections (Eq. (1)) and a dense
 * bf16 down projection W_down [E][I][H], the form whose down matrices the
 * paper leaves uncompressed (Sec. 3.1): routing as cardan_route_topk, g and
 * u as in cardan_vq_lr_expert_ffn, then y[t] = sum_j topk_w[t][j] *
 * W_down[e_j]^T p_j. The layer's cb_down, codes_down, A_down and B_down are
 * not read (may be NULL). Outputs as cardan_moe_layer. H * I * 2 must stay
 * below 2^31 (CARDAN_ERR_UNSUPPORTED otherwise). */
int cardan_moe_layer_dense_down(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                                const cardan_layer* layer, const cardan_bf16* W_down, float* y,
                                int32_t* topk_idx, float* topk_w,
                                void* ws, size_t ws_bytes, hipStream_t stream);

/* The uncompressed MoE layer (paper Sec. 2.1), the baseline the compressed
 * form is measured against: routing as cardan_route_topk, then for every
 * (token, selected expert) p = silu(W_gate[e]^T x) * (W_up[e]^T x) and
 * y[t] = sum_j topk_w[t][j] * W_down[e_j]^T p_j, float32 accumulation.
 * Only H, I, E and top_k of `shape` are read; the workspace size is
 * cardan_workspace_bytes() of any valid shape with those four fields.
 * H * I * 2 must stay below 2^31. Outputs as cardan_moe_layer. */
int cardan_dense_moe_layer(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                           const cardan_dense_layer* layer, float* y, int32_t* topk_idx,
                           float* topk_w, void* ws, size_t ws_bytes, hipStream_t stream);

/* The uncompressed layer with up-only squared-ReLU experts (Table 2, "up"):
 * as cardan_dense_moe_layer with p = max(W_up[e]^T x, 0)^2; W_gate is not
 * read (may be NULL). */
int cardan_dense_moe_layer_relu2(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                                 const cardan_dense_layer* layer, float* y, int32_t* topk_idx,
                                 float* topk_w, void* ws, size_t ws_bytes, hipStream_t stream);

/* RMS normalisation between stacked layers: x_next[t][h] =
 * bf16_rne(y[t][h] / sqrt(mean_h y[t][h]^2 + eps)), no learned scale.
 * y: [B][H] float32, x_next: [B][H] bf16. Needs no workspace. */
int cardan_rmsnorm_bf16(int32_t B, int32_t H, const float* y, float eps,
                        cardan_bf16* x_next, hipStream_t stream);

/* Kernel timing for measurement. cardan_profile_begin(n) makes the next n
 * calls launch each kernel with a HIP start/stop event pair recorded by the
 * dispatch itself (hipExtLaunchKernel), on the call's stream, so the pair
 * brackets the kernel's execution; cardan_profile_end() waits for those
 * events and writes, per
 * kernel kind, the summed milliseconds and the launch count (arrays of
 * length CARDAN_PROFILE_KINDS, ordered as the enum below). A layer call runs
 * the routing kernel (routing, shared projections, grouping) and then the
 * expert kernel (gate/up, down, combine). Host-global state: not
 * thread-safe, not for use under graph capture. */
enum {
  CARDAN_KERNEL_ROUTE = 0,    /* router, top-k, gating, grouping, z = U^T x */
  CARDAN_KERNEL_EXPERT = 1,   /* gate/up, down, weighted combine            */
  CARDAN_KERNEL_RMSNORM = 2,
  CARDAN_PROFILE_KINDS = 3
};
int cardan_profile_begin(int32_t max_calls);
int cardan_profile_end(float* ms_per_kind, int32_t* launches_per_kind);

#ifdef __cplusplus
}
#endif

#endif /* CARDAN_H */
