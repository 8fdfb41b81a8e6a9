/*
 * libgtr - chunkwise key-only gated linear attention (GLA) forward for MI355X
 * (gfx950), with the directional token-grid scans of the GTR backbone.
 *
 * Paper: "GTR" (arXiv 2609.26590).
 *   Sec. 3.1  "Key-only gated recurrence":  S_t = Diag(gamma_t) S_{t-1} + k_t^T v_t,
 *             o_t = d_k^{-1/2} q_t S_t, S_0 = 0, gamma_t in (0,1)^{d_k}.
 *   Sec. 3.1  "Directional scanning": one scan per block, left-to-right,
 *             right-to-left, top-to-bottom or bottom-to-top, with the spatial
 *             order restored afterwards.
 *   Sec. 3.3  "Hardware-Aware Chunkwise Inference", Eq. (chunk_boundary_main):
 *             chunk summaries U_c, decays d_c, boundary states
 *             S_[c+1] = Diag(d_c) S_[c] + U_c, and the chunk outputs.
 *   App. "Custom CUDA Operator": the operator consumes q, k, v and the
 *             log-decay g = log gamma; callers own persistent workspaces and
 *             preallocated outputs, and the calls are graph-capturable.
 *
 * Conventions for every entry point:
 *   - Tensor pointers are DEVICE pointers (hipMalloc'd or equivalent) unless
 *     stated otherwise; the argument struct itself is host memory.
 *   - The caller owns every buffer. The library never allocates, frees,
 *     synchronises, or copies between host and device on these calls, so they
 *     may be recorded into a HIP graph.
 *   - Arguments are validated on the host before any HIP call. On a nonzero
 *     status nothing has been launched and no buffer has been touched.
 *   - Kernels are enqueued on `stream`; results are valid once the stream has
 *     completed the work. A launch failure reported by the runtime maps to
 *     GTR_ERR_HIP.
 *   - All calls are thread-safe. The only state the library keeps between
 *     calls is a table of occupancy answers per (device, kernel), filled on
 *     first use under a lock and never changed afterwards; everything a call
 *     writes is in the caller's buffers.
 */
#ifndef GTR_H_
#define GTR_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GTR_OK = 0,
  GTR_ERR_NULL = 1,        /* a required pointer is NULL                          */
  GTR_ERR_SHAPE = 2,       /* a size is <= 0, a product overflows int64, (GLA)
                              one sequence's rows take 2 GB or more, or (SwiGLU)
                              a launch would need 2^31 work-groups or more        */
  GTR_ERR_UNSUPPORTED = 3, /* a dtype / head width / chunk / path not compiled in */
  GTR_ERR_ALIAS = 4,       /* an output overlaps an input or the workspace        */
  GTR_ERR_WORKSPACE = 5,   /* workspace missing, too small or not 256-B aligned   */
  GTR_ERR_HIP = 6,         /* the HIP runtime rejected a launch                   */
  GTR_ERR_SCRATCH = 7      /* (gtr_gla_fwd_noalloc) the call needs more workspace
                              than the library's fixed scratch holds            */
} gtr_status;

typedef enum { GTR_F32 = 0, GTR_F16 = 1, GTR_BF16 = 2 } gtr_dtype;

/*
 * Scan directions over an H x W token grid stored row-major (spatial index
 * i*W + j for row i, column j). pi(s) is the spatial index visited at scan
 * step s, L = H*W:
 *   GTR_SCAN_ROW      left-to-right: pi(s) = s
 *   GTR_SCAN_COL      top-to-bottom: s = j*H + i  ->  pi(s) = i*W + j
 *   GTR_SCAN_ROW_REV  right-to-left: pi(s) = L-1-s          (ROW reversed)
 *   GTR_SCAN_COL_REV  bottom-to-top: pi(s) = pi_COL(L-1-s)  (COL reversed)
 * The reversed scans are full reversals of the forward sequences.
 */
typedef enum {
  GTR_SCAN_ROW = 0,
  GTR_SCAN_COL = 1,
  GTR_SCAN_ROW_REV = 2,
  GTR_SCAN_COL_REV = 3
} gtr_scan;

/*
 * gtr_scan_permute - reorder token rows between spatial and scan order
 * (Sec. 3.1 "Directional scanning").
 *
 * src, dst : device, contiguous [outer, H*W, row_elems] elements of type `dt`.
 * inverse=0: dst[o, s, :] = src[o, pi(s), :]   (spatial -> scan order)
 * inverse=1: dst[o, pi(s), :] = src[o, s, :]   (scan order -> spatial)
 * A pure copy: the result is bit-exact. src and dst must not overlap
 * (GTR_ERR_ALIAS). outer >= 1, H >= 1, W >= 1, row_elems >= 1.
 */
gtr_status gtr_scan_permute(const void* src, void* dst, int64_t outer, int32_t H, int32_t W,
                            int64_t row_elems, gtr_dtype dt, gtr_scan dir, int32_t inverse,
                            hipStream_t stream);

/* What the g input of gtr_gla_fwd holds (Sec. 3.1, "Key-only gated recurrence":
 * the retention gate is gamma = sigmoid(a)^(1/tau) of a per-token, per-key-dim
 * logit a). */
typedef enum {
  GTR_GATE_LOG_DECAY = 0, /* g = log gamma, finite and <= 0 (the default)                */
  GTR_GATE_LOGITS = 1     /* g = a, any finite value; the kernels use
                             log gamma = logsigmoid(a) / gate_tau, in float32           */
} gtr_gate_kind;

/* Execution schedule of gtr_gla_fwd (all give the same result up to rounding;
 * the length-aware dispatch of the paper's operator appendix). */
typedef enum {
  GTR_PATH_AUTO = 0,   /* the library picks (gtr_gla_schedule reports the choice):
                          INLINE for sequences of at most 32 chunks whose chunks
                          are all resident at once; FUSED otherwise, up to 256
                          chunks for 16-bit inputs at chunk 64 and up to 64
                          chunks for the rest; STAGED beyond (or for more than
                          1024 sequences).                                          */
  GTR_PATH_FUSED = 1,  /* one launch, boundary states by look-back: each chunk
                          hands over its summary, finds S_[c] from the summaries
                          of the chunks before it back to the nearest chunk that
                          has handed over its inclusive state S_[j+1], and hands
                          over S_[c+1] in turn (the scan co-runs with the
                          outputs). For 16-bit inputs at chunk 64 and sequences
                          of more than 32 chunks the look-back goes by groups of
                          16 chunks: the last chunk of each group also hands over
                          the group's aggregate, and a chunk sums the summaries
                          of its own group and then one aggregate per earlier
                          group. At most 1024 sequences of 256 chunks.              */
  GTR_PATH_STAGED = 2, /* three launches: summaries, boundary-state scan, outputs;
                          no waits between work-groups                             */
  GTR_PATH_INLINE = 3  /* one launch, each chunk rebuilds its boundary state from
                          the summaries of all chunks before it (the paper's
                          inline prefixes for short sequences). Limits as FUSED.
                          With d_v = 64, no output gate and at most one
                          work-group per CU after doubling, the value columns of
                          each chunk are split over two work-groups (both
                          one-launch paths).                                       */
} gtr_path;

/*
 * Arguments of gtr_gla_fwd (host struct; pointers are device pointers).
 *
 * q, g : [B, heads, L, dk]   k : [B, heads, L, dk]   v : [B, heads, L, dv]
 *        contiguous, tokens in SPATIAL (row-major grid) order, L = H*W.
 *        g holds the log-decays g = log gamma (finite, <= 0); gamma = 1 is g = 0.
 *        A 1-D sequence is H = 1, W = L.
 * o    : [B, heads, L, dv] contiguous, written in SPATIAL order.
 * s0   : [B, heads, dk, dv] float32, the state before the first token in SCAN
 *        order; NULL means a zero state (the paper's S_0 = 0).
 * s_final : [B, heads, dk, dv] float32, receives the state after the last
 *        token in SCAN order; NULL means it is not written.
 * qkv_dtype : dtype of q, k, v.  g_dtype : qkv_dtype or GTR_F32.
 * o_dtype   : qkv_dtype or GTR_F32.
 * dk, dv : head widths; supported (dk, dv) = (32,32), (32,64), (64,64).
 * chunk  : chunk length C in {32, 64, 128} (Sec. 3.3; the paper uses 64).
 * scale  : o = scale * q S; the paper's value is dk^{-1/2}.
 * scan   : direction; the permutation is fused into the loads and stores.
 * path   : execution schedule (GTR_PATH_AUTO unless testing a schedule).
 * g_kind, gate_tau : gate fusion. With GTR_GATE_LOGITS, g holds the logits a
 *        of the retention gate and log gamma = logsigmoid(a) / gate_tau is
 *        formed in the kernels' loads (no separate pass over g).
 * out_gate, out_gate_dtype, norm_eps, norm_weight : output-gate epilogue
 *        (Sec. 3.1: u_t = SiLU(x_t W_r) * RMSNorm(o_t); the operator appendix
 *        fuses it into the output kernel). When out_gate is not NULL it holds
 *        x W_r in SPATIAL order like o, and o receives, per token and head,
 *          u_j = SiLU(z_j) * o_j / sqrt(mean_i o_i^2 + norm_eps) * w_j,
 *        mean over the dv channels of that head, o the scaled output above,
 *        z = out_gate, w = norm_weight (ones if NULL); float32 arithmetic.
 *        out_gate must not overlap o.
 * workspace, workspace_bytes : device scratch owned by the caller, at least
 *        gtr_gla_workspace_size(args) bytes, 256-byte aligned, and zero-filled
 *        before its first use (gtr_gla_workspace_init). Its first 32-bit word
 *        is the fault word (below). The synchronisation words of the one-launch
 *        schedules sit in regions of fixed place and size that no other part of
 *        any call's workspace overlaps, and every completed call leaves them
 *        zeroed again, so one workspace (large enough for each) serves any
 *        number of calls of any shapes on one stream. Calls that overlap in
 *        time (two streams, for instance) must not share a workspace.
 * spin_limit : polls a one-launch work-group makes while it waits for the
 *        chunks before it, before it gives up (0: the library default, about a
 *        second). A work-group that gives up sets bit 0 of the fault word and
 *        writes NaN into its output rows, into the state it hands over (so
 *        every chunk after it is NaN too) and into S_final where it writes it;
 *        every work-group still exits normally. Outputs that are not NaN are
 *        valid. A small limit forces the condition (tests).
 *
 * Fault word (stream-ordered status, sticky until gtr_gla_workspace_init):
 *   bit 0  a bounded wait ran out (see spin_limit);
 *   bit 1  a bf16 q, k or v value lies outside the fp16 range (|x| > 65504):
 *          the work-groups that read it write NaN in its chunk's output rows
 *          (and, in the one-launch schedules, in everything after it).
 * Read it with gtr_gla_workspace_fault after the stream has completed the call.
 *
 * Numerics: float32 accumulation throughout. With fp16/bf16 inputs the matrix
 * products use fp16 operands: the rescaled q and k are bounded by |q| and |k|,
 * and the score tile, the chunk summaries and the boundary states are scaled
 * by powers of two before they are rounded to fp16, so no intermediate
 * overflows for inputs within the fp16 range (bf16 inputs are checked, above).
 * With float32 inputs every product is float32. Inputs must be finite.
 */
typedef struct {
  const void* q;
  const void* k;
  const void* v;
  const void* g;
  void* o;
  const float* s0;
  float* s_final;
  gtr_dtype qkv_dtype;
  gtr_dtype g_dtype;
  gtr_dtype o_dtype;
  int32_t B, heads, H, W;
  int32_t dk, dv, chunk;
  float scale;
  gtr_scan scan;
  gtr_path path;
  void* workspace;
  size_t workspace_bytes;
  /* Optional fusions; a zero-initialised struct leaves both off. */
  gtr_gate_kind g_kind;     /* what g holds (gtr_gate_kind)                           */
  float gate_tau;           /* GTR_GATE_LOGITS: the temperature tau (> 0; paper: 16)  */
  const void* out_gate;     /* [B, heads, L, dv] output-gate pre-activation x W_r, or
                               NULL for no epilogue                                   */
  gtr_dtype out_gate_dtype; /* qkv_dtype or GTR_F32                                   */
  float norm_eps;           /* RMSNorm epsilon (> 0) of the epilogue                  */
  const float* norm_weight; /* [dv] RMSNorm weight, or NULL for ones                  */
  uint32_t spin_limit;      /* bounded-wait polls of the one-launch schedules; 0 = default */
} gtr_gla_args;

/* Bytes of workspace gtr_gla_fwd needs for these arguments (host only, no HIP
 * call). Returns 0 if the arguments are invalid. Pointer fields are ignored. */
size_t gtr_gla_workspace_size(const gtr_gla_args* args);

/* Zero-fill `bytes` bytes of a workspace with a kernel on `stream` (no memset
 * node, so it may be recorded into a graph). */
gtr_status gtr_gla_workspace_init(void* workspace, size_t bytes, hipStream_t stream);

/*
 * gtr_gla_fwd - chunkwise key-only GLA forward (Sec. 3.1 recurrence evaluated
 * with the chunkwise schedule of Sec. 3.3), scanning in direction `scan`.
 * For every (b, h): visiting tokens in scan order, S = s0 (or 0),
 *   S <- Diag(exp(g_t)) S + k_t^T v_t,   o_t = scale * q_t S,
 * with o written back at the token's spatial index, and S_final = S at the end.
 */
gtr_status gtr_gla_fwd(const gtr_gla_args* args, hipStream_t stream);

/*
 * gtr_gla_schedule - the schedule gtr_gla_fwd would run for `args`
 * (GTR_PATH_FUSED, GTR_PATH_STAGED or GTR_PATH_INLINE; for an explicit path,
 * that path), or -1 if the arguments are invalid (pointers are not checked) or
 * an explicit one-launch path does not fit. Host-only; reads the current
 * device's occupancy for the one-launch schedules (without a usable device
 * AUTO reports GTR_PATH_STAGED). The length-aware dispatch of the paper's
 * operator appendix.
 */
int gtr_gla_schedule(const gtr_gla_args* args);

/*
 * gtr_gla_value_parts - how many work-groups share each chunk's d_v value
 * columns in the schedule gtr_gla_schedule reports: 2 where the inline
 * schedule splits them (d_v = 64, no output gate, and at most one work-group
 * per CU after doubling), else 1; -1 where gtr_gla_schedule gives -1.
 * Host-only, like gtr_gla_schedule. The split changes which work-group
 * computes what, not the arithmetic of any output element.
 */
int gtr_gla_value_parts(const gtr_gla_args* args);

/*
 * Spatial SwiGLU (Sec. 3.1, "Spatial SwiGLU"):
 *   Y = [SiLU(X W_g) * DWConv3x3(X W_v)] W_o
 * for every image b: X = x[b] is [H*W, d] in SPATIAL (row-major grid) order, the
 * value branch X W_v is convolved depthwise over the H x W grid (3 x 3,
 * cross-correlation, zero padding, optional bias), the gate is tokenwise.
 *
 * x       : [B, H*W, d]           dtype
 * w_gate  : [hidden, d]           dtype (linear-layer layout, output features first)
 * w_value : [hidden, d]           dtype
 * w_out   : [d, hidden]           dtype
 * conv_w  : [hidden, 3, 3]        float32, conv_w[c][u][v] weighs the token at
 *                                 grid offset (u - 1, v - 1)
 * conv_b  : [hidden] float32 or NULL
 * y       : [B, H*W, d]           y_dtype (dtype or GTR_F32); must not overlap
 *                                 the inputs or the workspace; y = residual + Y
 *                                 when residual (below) is not NULL
 * dtype   : GTR_F16 or GTR_BF16; d and hidden multiples of 64; every pointer
 *           16-byte aligned.
 * The products accumulate in float32; X W_g and X W_v are rounded to fp16 on
 * chip (one launch forms the gated convolution per tile of tokens, its halo
 * recomputed), the gated hidden activations are stored in fp16 for the output
 * product; all three must stay finite in fp16.
 * workspace : caller-owned, 256-byte aligned, gtr_spatial_swiglu_workspace_size
 *           bytes (B*H*W*hidden*2 for the activations plus the float32 partial
 *           products of a K-split output product, rounded up); no
 *           initialisation needed.
 * Errors as for gtr_gla_fwd; every check runs before any launch.
 */
typedef struct {
  const void* x;
  const void* w_gate;
  const void* w_value;
  const void* w_out;
  const float* conv_w;
  const float* conv_b;
  void* y;
  gtr_dtype dtype;
  gtr_dtype y_dtype;
  int32_t B, H, W, d, hidden;
  void* workspace;
  size_t workspace_bytes;
  const void* residual;  /* [B, H*W, d] in y_dtype added to y (a block's residual), or NULL; may be y itself */
} gtr_swiglu_args;

size_t gtr_spatial_swiglu_workspace_size(const gtr_swiglu_args* args);
gtr_status gtr_spatial_swiglu(const gtr_swiglu_args* args, hipStream_t stream);

/*
 * The remaining entry points serve one GTR block (Sec. 3.1: projections, the
 * key-only gated recurrence with its output gate, head concat and W_o, then
 * Spatial SwiGLU), composed from them and the calls above.
 *
 * gtr_gemm: C = A B^T (+ bias) (+ res), the block's projections. a and c may
 * be head-major (a_tokens, c_tokens below; zero for row-major).
 * a       : [M, K] row-major, a_dtype (GTR_F16 or GTR_BF16)
 * b       : [N, K] row-major (linear-layer weight layout, output features
 *           first), b_dtype = a_dtype
 * c       : [M, N] row-major, c_dtype (GTR_F32, GTR_F16 or GTR_BF16); must not
 *           overlap a, b or bias
 * bias    : [N] float32 added to every row, or NULL
 * res     : [M, N] in c_dtype added elementwise (a residual), or NULL; may be c
 *           itself (in place), must not overlap it otherwise
 * row_norm: 0, or 1 to normalise every row of a over its K columns first:
 *           C = ((A - mu) / sqrt(var + row_norm_eps)) B^T (+ bias) (+ res),
 *           mu and var the mean and biased variance of the row (float32). A
 *           layer normalisation with weights gamma, beta before a linear layer
 *           W, bias c is this call with b = W diag(gamma) and bias = c + W beta
 *           (Sec. 3.1's pre-norm block). Needs a row-major a (a_tokens 0) and
 *           0 <= row_norm_eps < 1e30.
 * N and K multiples of 64, every pointer 16-byte aligned. The products
 * accumulate in float32 (MFMA on the input dtype) and are rounded once into c.
 * Errors as for gtr_gla_fwd; every check runs before the launch.
 */
typedef struct {
  const void* a;
  const void* b;
  void* c;
  const float* bias;
  const void* res;
  gtr_dtype a_dtype, b_dtype, c_dtype;
  int64_t M;
  int32_t N, K;
  int64_t a_tokens;    /* 0, or a head-major a: [M / a_tokens][K / 64][a_tokens][64], row m = token m % a_tokens
                          of image m / a_tokens, columns 64 h .. 64 h + 63 = head h (a head concat read in
                          place; M a multiple of a_tokens) */
  int64_t c_tokens;    /* 0, or a head-major c: [N / (c_heads c_head_dim)][M / c_tokens][c_heads][c_tokens]
                          [c_head_dim] (projections split into heads as they are stored; M a multiple of
                          c_tokens, N of c_heads c_head_dim, c_head_dim of 4, res NULL) */
  int32_t c_heads, c_head_dim;
  float row_norm_eps;  /* the row normalisation's epsilon (row_norm 1) */
  int32_t row_norm;    /* 0, or 1: normalise the rows of a (above) */
} gtr_gemm_args;

gtr_status gtr_gemm(const gtr_gemm_args* args, hipStream_t stream);

/*
 * gtr_layernorm: y[m] = (x[m] - mean) / sqrt(var + eps) * w + b over the d
 * channels of every row m (mean and biased variance of the row, in float32).
 * x, y : [M, d] dtype (GTR_F16 or GTR_BF16); y may be x (in place).
 * w, b : [d] float32; NULL stands for ones / zeros.
 * d a multiple of 8 and at most 2048; x, y, w, b 16-byte aligned.
 */
gtr_status gtr_layernorm(const void* x, const float* w, const float* b, void* y, int64_t M, int32_t d, float eps,
                         gtr_dtype dtype, hipStream_t stream);

/*
 * gtr_heads_split: the columns of a token-major product into head-major
 * tensors, as the GLA call takes them.
 *   src : [B*L, ld] dtype; part p, head h is columns p*H*dh + h*dh .. + dh - 1
 *   dst : [parts][B][H][L][dh] dtype, contiguous
 * gtr_heads_merge: the reverse for one part: src [B][H][L][dh] ->
 *   dst [B*L][H*dh].
 * dtype GTR_F16 or GTR_BF16; dh a multiple of 8; ld >= parts*H*dh and a
 * multiple of 8; src and dst 16-byte aligned and not overlapping.
 */
gtr_status gtr_heads_split(const void* src, void* dst, int32_t parts, int32_t B, int32_t H, int64_t L, int32_t dh,
                           int64_t ld, gtr_dtype dtype, hipStream_t stream);
gtr_status gtr_heads_merge(const void* src, void* dst, int32_t B, int32_t H, int64_t L, int32_t dh, gtr_dtype dtype,
                           hipStream_t stream);

/*
 * gtr_add: y = a + b elementwise over n elements (a residual), rounded once
 * into dtype (GTR_F16 or GTR_BF16). n a multiple of 8; pointers 16-byte
 * aligned; y may be a or b.
 */
gtr_status gtr_add(const void* a, const void* b, void* y, int64_t n, gtr_dtype dtype, hipStream_t stream);

/*
 * gtr_gla_fwd_noalloc - gtr_gla_fwd for callers that cannot allocate device
 * memory (code under HIP graph capture, serving loops, harnesses that forbid
 * hipMalloc). Same arguments, results and schedules as gtr_gla_fwd, except
 * that args->workspace and args->workspace_bytes are ignored: the workspace is
 * a fixed 32 MB scratch array inside the library, one copy per device, held
 * until the process ends. The call itself allocates and frees nothing and
 * calls no allocating routine; the first call on a device looks up that
 * device's copy of the array (hipGetSymbolAddress), once.
 * A call that needs more than 32 MB of workspace (gtr_gla_workspace_size) is
 * rejected with GTR_ERR_SCRATCH before anything is launched; this holds the
 * 40x40-token workloads up to 16 sequences and 6 sequences at 80x80, for
 * instance, not a batch of 8 images of 12 heads.
 * Every call on a device shares that device's array: calls that overlap in
 * time on one device (two streams, two threads) race and must not be issued.
 * The scratch keeps what the last call left: its synchronisation words are
 * zero at load and every completed call leaves them zero. Its fault word
 * cannot be read through this interface; a wait that ran out still shows as
 * NaN in the outputs it poisoned.
 */
gtr_status gtr_gla_fwd_noalloc(const gtr_gla_args* args, hipStream_t stream);

/* The fault word of a workspace (bits as described under gtr_gla_args: 1 = a
 * bounded wait ran out, 2 = a bf16 input outside the fp16 range), 0 if every
 * call since the last gtr_gla_workspace_init was clean. Reads it with a
 * blocking device-to-host copy, so call it after the stream has completed the
 * calls of interest - a check for tests and for callers that can afford a
 * synchronisation, not for the hot path. Returns -1 on a HIP error. */
int gtr_gla_workspace_fault(const void* workspace, size_t bytes);

const char* gtr_status_string(gtr_status status);

#ifdef __cplusplus
}
#endif

#endif /* GTR_H_ */
