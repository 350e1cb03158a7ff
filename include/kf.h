/*
 * kf.h -- C ABI of libkf.so: fused contraction + epilogue chains on AMD
 * MI355X (gfx950).
 *
 * An operation is a dense contraction followed by an ordered list of
 * epilogue ops, executed as one kernel (plus, for row-wise softmax and
 * logsumexp over more columns than one tile holds, a short finishing
 * kernel).  This is the computation the paper's search turns into single
 * kernels: a PyTorch operator given as a reference computation (Methodology,
 * Overview) rewritten by operator fusion -- matmul + activation,
 * normalisation + activation, softmax -- and by reduced precision and online
 * softmax (Appendix A, allowed optimisation strategies).  The op descriptor
 * mirrors that problem statement: the reference module's contraction, its
 * parameters in module order, and its forward's op sequence.
 *
 * Conventions
 *   - All tensors are device memory (hipMalloc'd or torch-allocated) owned
 *     by the caller; the library never frees or reallocates them.
 *   - Strides are in elements.  The innermost stride must be 1 (the
 *     channels-last KF_CONV3D_3X3X3 input is the one exception, described
 *     there) and every base pointer 16-byte aligned (the kernels use 128-bit
 *     loads).
 *   - `stream` is a hipStream_t passed as void* (NULL = default stream).
 *     Calls are asynchronous: launch errors are returned, device faults
 *     surface at the caller's next synchronisation on that stream.
 *   - No function aborts or throws; every failure returns a kf_status and
 *     kf_last_error() (thread-local) describes it.
 *   - Accumulation is always fp32.
 *   - Nothing in the measured path calls rocBLAS, hipBLASLt, MIOpen or a
 *     PyTorch op: every step runs in this library's own kernels.
 */
#ifndef KF_H_
#define KF_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum kf_status {
  KF_OK = 0,
  KF_ERR_INVALID_ARG = 1,  /* NULL pointer, bad enum value, bad count        */
  KF_ERR_SHAPE = 2,        /* tensor shape/dtype/stride disagrees with spec  */
  KF_ERR_UNSUPPORTED = 3,  /* well-formed but not implemented (e.g. a row op
                              not last, misaligned pointer, K % 8 != 0)      */
  KF_ERR_NO_DEVICE = 4,    /* no usable gfx950 device                        */
  KF_ERR_OOM = 5,          /* workspace allocation failed                    */
  KF_ERR_HIP = 6           /* a HIP runtime call failed                      */
} kf_status;

typedef enum kf_contraction {
  /* h[m][n] = sum_k A[m][k] * B(k, n); A is [M,K] row-major, B is [K,N]
     (KF_LAYOUT_KN) or [N,K] (KF_LAYOUT_NK, nn.Linear's weight layout). */
  KF_GEMM = 0,
  /* PyTorch Conv2d (cross-correlation), 3x3 kernel, stride 1, zero padding
     1, dilation 1, groups 1.  A = input [batch,cin,H,W] (NCHW), B = weight
     [cout,cin,3,3] (OIHW); h is [batch,cout,H,W]. */
  KF_CONV2D_3X3 = 1,
  /* No contraction: h = A, an [M,N] row-major tensor (fp32 or bf16, any row
     stride), and the op list runs over its rows -- the memory-bound
     reduction chains (softmax, logsumexp, GroupNorm with their element-wise
     neighbours).  No B input; K is ignored.  N % 8 == 0; N <= 16384, except
     for a list that ends with ROW_LOGSUMEXP or ROW_CROSS_ENTROPY after only
     BIAS and element-wise ops (rows streamed: N < 2^31); GROUPNORM needs
     (N / groups) % 8 == 0. */
  KF_ROWWISE = 2,
  /* PyTorch Conv3d (3-D cross-correlation), 3x3x3 kernel, stride 1, no
     padding (Conv3d's default), dilation 1, groups 1 -- the convolution of
     the Conv3d -> softmax -> max-pool operator in the paper's case study
     (Appendix C).  A = input [batch,cin,depth,height,width] stored
     channels-last (torch.channels_last_3d: strides [D*H*W*cin, 1, H*W*cin,
     W*cin, cin]) or contiguous NCDHW; B = weight [cout,cin,3,3,3] contiguous
     (OIDHW); h is [batch,cout,depth-2,height-2,width-2].  bf16 in and out.
     cin = 16, cout = 64 with a channels-last input runs the tiled kernel,
     which fuses the whole op list, CHANNEL_SOFTMAX and MAXPOOL3D_2 included
     (the whole channel axis in one tile, so the channel softmax is
     tile-local).  Any other cin, cout or layout runs the general kernel,
     which fuses the leading BIAS and element-wise ops; a CHANNEL_SOFTMAX or
     MAXPOOL3D_2 and every op after it then run partly fused: one kernel per
     op over bf16 intermediates in two buffers the descriptor allocates on
     the first such call (2 x batch x cout x (depth-2)(height-2)(width-2)
     bf16; KF_ERR_OOM if that fails), which kf_fused_op_noalloc refuses. */
  KF_CONV3D_3X3X3 = 3
} kf_contraction;

typedef enum kf_dtype {
  KF_F32 = 0,
  KF_BF16 = 1,
  KF_FP8_E4M3 = 2, /* OCP E4M3 (bias 7, max 448, no Inf); GEMM only, with
                      per-tensor fp32 scales: A_real = dec(A) * scale_a. */
  KF_I32 = 3       /* int32: the class targets of ROW_CROSS_ENTROPY only   */
} kf_dtype;

typedef enum kf_layout { KF_LAYOUT_KN = 0, KF_LAYOUT_NK = 1 } kf_layout;

/* Epilogue ops, applied in list order to the fp32 contraction result.
   "feature" means the GEMM output column n, or the conv output channel. */
typedef enum kf_op_kind {
  KF_OP_BIAS = 1,          /* h += bias[feature]          (input fp32 [F])  */
  KF_OP_RELU = 2,          /* max(h, 0)                                     */
  KF_OP_GELU_TANH = 3,     /* 0.5 h (1 + tanh(sqrt(2/pi)(h + 0.044715 h^3))) */
  KF_OP_GELU_ERF = 4,      /* 0.5 h (1 + erf(h / sqrt 2))                    */
  KF_OP_SWISH = 5,         /* h * sigmoid(h)                                */
  KF_OP_SIGMOID = 6,       /* 1 / (1 + e^-h)                                */
  KF_OP_TANH = 7,          /* tanh(h)                                       */
  KF_OP_HARDTANH = 8,      /* clamp(h, p0, p1)                              */
  KF_OP_SCALE = 9,         /* h * p0                                        */
  KF_OP_GROUPNORM = 10,    /* nn.GroupNorm over features: `groups` groups of
                              contiguous features per row, biased variance,
                              eps = p0, then gamma/beta affine
                              (inputs fp32 [F] each). GEMM or ROWWISE.     */
  KF_OP_RESIDUAL_ADD = 11, /* h += residual (input, same shape as output;
                              dtype = spec.residual_dtype)                  */
  KF_OP_MAXPOOL2X2 = 12,   /* MaxPool2d(2, stride 2) on the conv output;
                              CONV2D only, H and W even. Output shape
                              [batch,cout,H/2,W/2].                         */
  KF_OP_ROW_SOFTMAX = 13,  /* softmax over the last axis; GEMM or ROWWISE;
                              last op                                       */
  KF_OP_ROW_LOGSUMEXP = 14,/* log sum exp over the last axis; GEMM or
                              ROWWISE; last op; output becomes fp32 [M]     */
  KF_OP_CHANNEL_SOFTMAX = 15,/* softmax over the output channels at every
                              position (torch.softmax(h, dim=1));
                              CONV3D_3X3X3 only, at most once               */
  KF_OP_MAXPOOL3D_2 = 16,  /* MaxPool3d(2): kernel 2, stride 2, no padding,
                              floor mode; CONV3D_3X3X3 only, after every
                              other op.  The fused kernel takes zero or two
                              of them (two in a row = one max over aligned
                              4x4x4 blocks).                                */
  KF_OP_ROW_CROSS_ENTROPY = 17 /* nn.CrossEntropyLoss(reduction='none') with
                              class-index targets: loss_m = logsumexp_n h[m][n]
                              - h[m][t_m] (the loss operators of the paper's
                              reduction categories, Table 2); GEMM or ROWWISE;
                              last op; input int32 targets [M] (KF_I32), each
                              in [0, N) -- a target outside gives NaN; output
                              fp32 [M]                                      */
} kf_op_kind;

typedef struct kf_op {
  int32_t kind;    /* kf_op_kind                                            */
  int32_t groups;  /* GROUPNORM: number of groups                           */
  float p0;        /* HARDTANH lo, SCALE factor, GROUPNORM eps              */
  float p1;        /* HARDTANH hi                                           */
} kf_op;

#define KF_MAX_OPS 8

typedef struct kf_op_spec {
  int32_t contraction;     /* kf_contraction                                */
  int32_t in_dtype;        /* kf_dtype of A and B                           */
  int32_t out_dtype;       /* KF_F32 or KF_BF16 (ROW_LOGSUMEXP: KF_F32)      */
  int32_t b_layout;        /* kf_layout (GEMM)                              */
  int64_t M, N, K;         /* GEMM sizes                                    */
  int64_t batch, cin, height, width, cout; /* CONV2D_3X3 / CONV3D sizes     */
  int64_t depth;           /* CONV3D_3X3X3 input depth                      */
  float scale_a, scale_b;  /* FP8_E4M3 per-tensor dequantisation scales     */
  int32_t residual_dtype;  /* KF_F32 or KF_BF16, for RESIDUAL_ADD           */
  int32_t n_ops;           /* 0..KF_MAX_OPS                                 */
  kf_op ops[KF_MAX_OPS];
} kf_op_spec;

#define KF_MAX_DIMS 5

typedef struct kf_tensor {
  void* data;              /* device pointer, 16-byte aligned               */
  int32_t dtype;           /* kf_dtype                                      */
  int32_t ndim;            /* 1..KF_MAX_DIMS                                */
  int64_t shape[KF_MAX_DIMS];
  int64_t stride[KF_MAX_DIMS]; /* elements; stride[ndim-1] must be 1, except
                              for the channels-last CONV3D input            */
} kf_tensor;

typedef struct kf_desc kf_desc;

/* Validate `spec` and plan the operation: kernel variant, tile shape and a
   device workspace (owned by the descriptor) for the repacked conv weights or
   the cross-tile row partials.  The spec is the paper's problem statement of
   an operator given as a PyTorch reference computation (Methodology,
   Overview): the contraction, its shapes and dtypes, and the forward's op
   sequence, parameters in module order.
   Validation happens on the host before any device call, so spec errors are
   reported (KF_ERR_INVALID_ARG / _SHAPE / _UNSUPPORTED) even with no GPU
   present; a valid spec with no gfx950 device returns KF_ERR_NO_DEVICE, a
   failed workspace allocation KF_ERR_OOM.  On any error *out is set to NULL.
   The caller owns *out and frees it with kf_destroy. */
kf_status kf_create(const kf_op_spec* spec, kf_desc** out);

/* Run the fused operation on `stream`: the contraction and the whole op list
   in one kernel, intermediates kept in registers (the operator fusion and
   online softmax of Appendix A), plus, for a row softmax / logsumexp over
   more than one 256-column tile, a finishing kernel over the per-tile
   partials (Appendix B, hierarchical reductions).
   inputs (in this order): A, B (no B for KF_ROWWISE), then one slot per
   tensor the ops need, in op order -- BIAS: bias; GROUPNORM: gamma, beta;
   RESIDUAL_ADD: residual; ROW_CROSS_ENTROPY: targets.  All are device
   pointers owned by the caller.
   outputs: exactly one tensor (shape from kf_output_info, dtype
   spec.out_dtype), written, never reallocated.
   Returns KF_ERR_SHAPE / _UNSUPPORTED / _INVALID_ARG when a tensor does not
   match the plan (nothing is launched), KF_ERR_HIP when a launch fails.  The
   descriptor's workspace is reused by every call, so at most one call per
   descriptor may be in flight at a time (use one descriptor per stream).
   Conv plans repack B into the workspace on the first call and again only
   when B's data pointer changes: after rewriting B's contents in place, call
   kf_weights_changed first.  After one call on the same tensors the call
   enqueues kernels only (no allocation, memset or synchronisation), so it
   can be recorded in a HIP graph and replayed (a Conv3d chain that runs
   partly fused allocates its intermediates on that first call). */
kf_status kf_fused_op(const kf_desc* desc, const kf_tensor* inputs,
                      kf_tensor* outputs, void* stream);

/* kf_fused_op, additionally recording `ev_before` and `ev_after` (hipEvent_t
   created by the caller, passed as void*) on `stream` immediately before and
   after the main contraction kernel, so that hipEventElapsedTime gives that
   kernel's duration alone (finishing kernels, and the per-op kernels of a
   partly fused Conv3d chain, fall outside the pair).  Either
   event may be NULL. */
kf_status kf_fused_op_timed(const kf_desc* desc, const kf_tensor* inputs,
                            kf_tensor* outputs, void* stream, void* ev_before,
                            void* ev_after);

/* Declare that the contents of the weight tensor B changed in place since
   the last call: the next call of a conv plan repacks it.  (A different B
   pointer is noticed without this.)  NULL is a no-op. */
void kf_weights_changed(kf_desc* desc);

/* Clock stamps of the bf16 / fp8 GEMM kernel, for the diagnosis (which rests
   on knowing what the kernel ran at and where its time goes, Methodology,
   Diagnosis): after this call, every launch of the plan's 256x256 kernel
   (launch variants 0 and 2) writes, for each workgroup b < `workgroups`, six
   int64 values to stamps[6b .. 6b+5]: c0, c1 = the shader-clock counter at
   the workgroup's start and end; w0, w1 = the constant-rate counter
   (kf_wall_clock_hz) at its start and end; cp, ck = the shader-clock counter
   when the first operand stage has landed (end of the prologue) and when
   the K loop has ended (its last stage drained, before the epilogue).  So
   (c1 - c0) / ((w1 - w0) / rate) is the shader clock the tile ran at,
   (w1 - w0) / rate its duration, and cp - c0, ck - cp, c1 - ck the shader
   cycles of prologue, K loop and epilogue.  Workgroup b computes one
   256x256 output tile.  `stamps` is a device buffer of at least
   6 x workgroups int64, 8-byte aligned, owned by the caller; NULL turns the
   stamps off.  The 128x256 kernel (variant 1) records none.  Errors:
   KF_ERR_UNSUPPORTED for other plans, KF_ERR_INVALID_ARG. */
kf_status kf_set_clock_stamps(kf_desc* desc, void* stamps, int64_t workgroups);

/* The frequency of the constant-rate counter of the current device in Hz
   (the rate of the stamps' w values), or -1 without a device. */
int64_t kf_wall_clock_hz(void);

/* The same operation as an unfused chain, one kernel per op, with every
   intermediate stored to device memory in bf16 (fp32 for fp32 chains) --
   the one-operator-per-kernel form that operator fusion removes (Appendix A,
   "Operator Fusion"), the comparator for the fused kernel.  Its
   intermediate buffers are allocated on the first call and owned by the
   descriptor (KF_ERR_OOM if that fails); errors as for kf_fused_op. */
kf_status kf_unfused_op(const kf_desc* desc, const kf_tensor* inputs,
                        kf_tensor* outputs, void* stream);

/* Free the workspace and the descriptor.  NULL is a no-op.  The caller must
   make sure no call using `desc` is still running. */
void kf_destroy(kf_desc* desc);

/* Number of input slots the operation expects. */
int32_t kf_num_inputs(const kf_desc* desc);

/* Expected dtype / shape of input slot `slot`, and of the single output. */
kf_status kf_input_info(const kf_desc* desc, int32_t slot, int32_t* dtype,
                        int32_t* ndim, int64_t shape[KF_MAX_DIMS]);
kf_status kf_output_info(const kf_desc* desc, int32_t* dtype, int32_t* ndim,
                         int64_t shape[KF_MAX_DIMS]);

/* Bytes of device workspace the descriptor owns (fused path). */
size_t kf_workspace_bytes(const kf_desc* desc);

/* Name of the main kernel the plan launches (the contraction, or the row
   kernel of a ROWWISE list) under its current launch configuration; a
   static string. */
const char* kf_kernel_name(const kf_desc* desc);

/* ---- Diagnosis and tuning ------------------------------------------------
   The deterministic core of the paper's diagnosis engine (Methodology,
   Diagnosis and Experience-Guided Feedback): from runtime statistics and the
   kernel's launch configuration a correct kernel is classified as
   memory-bound, latency-bound or instruction-bound, and the launch fields of
   the plan are then searched by timing, keeping the fastest -- the paper's
   recommendations for such kernels are to autotune tile shapes and the
   mapping of work to programs, and to keep accesses local to the caches
   (Appendix B, latency-bound and memory-bound lists). */

typedef enum kf_bound {
  KF_BOUND_MEMORY = 0,      /* the HBM roof is the nearer one                 */
  KF_BOUND_INSTRUCTION = 1, /* the arithmetic (matrix-core / vector) roof is
                               the nearer one                                 */
  KF_BOUND_LATENCY = 2      /* neither roof is approached, or the launch has
                               fewer workgroups than compute units           */
} kf_bound;

typedef struct kf_diagnosis {
  double flops;         /* algorithmic FLOPs of the main kernel (2 per MAC)  */
  double bytes;         /* HBM bytes: the measured count if one was given,
                           else the algorithmic bytes (each input read once,
                           the output written once)                         */
  double seconds;       /* the main kernel's duration                        */
  double tflops;        /* flops / seconds / 1e12                            */
  double gbps;          /* bytes / seconds / 1e9                             */
  double peak_tflops;   /* dense peak of the kernel's arithmetic on MI355X   */
  double peak_gbps;     /* HBM peak of MI355X (8000)                         */
  double compute_frac;  /* tflops / peak_tflops                              */
  double memory_frac;   /* gbps / peak_gbps                                  */
  double intensity;     /* flops / bytes                                     */
  double ridge;         /* peak FLOP/s / peak byte/s                         */
  int64_t workgroups;   /* workgroups the main kernel launches               */
  int32_t compute_units;
  int32_t bound;        /* kf_bound                                          */
  double mfma_busy;     /* counted matrix-core busy fraction (-1: not given) */
  double lds_conflict;  /* counted LDS bank-conflict share of LDS-active
                           cycles (-1: not given)                           */
  double traffic_ratio; /* counted HBM bytes / algorithmic bytes (-1: no
                           count given)                                     */
  uint32_t hints;       /* kf_hint bits: what to change, by the rules of
                           kf_diagnose_counters                             */
  int32_t reserved;     /* 0                                                 */
} kf_diagnosis;

/* Recommendations a diagnosis can carry (bits of kf_diagnosis.hints): the
   paper's expert advice per bottleneck class (Appendix B), keyed on
   counted evidence. */
typedef enum kf_hint {
  KF_HINT_REUSE = 1,        /* HBM traffic well above the algorithmic bytes:
                               improve operand reuse (tile order / raster,
                               keep data resident in LDS or registers)       */
  KF_HINT_PARALLELISM = 2,  /* fewer workgroups than compute units: split the
                               work finer or process more per launch         */
  KF_HINT_PIPELINE = 4,     /* latency-bound: deepen prefetch / pipelining,
                               raise the bytes in flight                      */
  KF_HINT_OVERLAP = 8,      /* instruction-bound with the matrix cores idle
                               much of the time: overlap loads, barriers and
                               the epilogue with the MFMA work               */
  KF_HINT_LDS_LAYOUT = 16   /* LDS bank conflicts: change the LDS layout or
                               swizzle                                       */
} kf_hint;

/* The classification rule alone (no descriptor, no device): latency-bound if
   workgroups < compute_units or both fractions are below 0.25, else
   memory-bound if memory_frac >= compute_frac, else instruction-bound.
   Fills every field of *out from the arguments; seconds must be > 0. */
kf_status kf_classify(double flops, double bytes, double seconds, double peak_tflops, double peak_gbps,
                      int64_t workgroups, int32_t compute_units, kf_diagnosis* out);

/* Diagnose a planned op from a measured main-kernel duration (for instance
   the event pair of kf_fused_op_timed) and, if hbm_bytes > 0, a measured HBM
   byte count (e.g. the FETCH_SIZE + WRITE_SIZE counters of one launch);
   hbm_bytes <= 0 uses the algorithmic bytes of the plan. */
kf_status kf_diagnose(const kf_desc* desc, double kernel_seconds, double hbm_bytes, kf_diagnosis* out);

/* Hardware counters of one launch of the plan's main kernel, as rocprofv3
   reports them (each field < 0 when not measured, except kernel_seconds). */
typedef struct kf_counters {
  double kernel_seconds;   /* duration of the launch, > 0                    */
  double hbm_bytes;        /* FETCH_SIZE + WRITE_SIZE, scaled to bytes by a
                              plain-copy calibration                         */
  double mfma_busy;        /* SQ_VALU_MFMA_BUSY_CYCLES / (SIMDs x per-XCD
                              GRBM_GUI_ACTIVE): 0..1                         */
  double lds_conflict;     /* SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE: 0..1 */
} kf_counters;

/* kf_diagnose from counters: the compute fraction is the counted
   matrix-core busy fraction when it is given (for matrix-core kernels; the
   achieved FLOP rate over the datasheet peak otherwise), the memory fraction
   the counted bytes over the HBM peak; the bound then follows kf_classify's
   rule, and the hints are set as: REUSE if counted bytes exceed 1.5x the
   algorithmic bytes of a memory-bound or matrix-core kernel; PARALLELISM if
   fewer workgroups than compute units; PIPELINE if latency-bound; OVERLAP
   if instruction-bound with the matrix cores busy less than 75% of the
   cycles; LDS_LAYOUT if more than 5% of the LDS-active cycles are bank
   conflicts.  The thresholds are this library's, not the paper's. */
kf_status kf_diagnose_counters(const kf_desc* desc, const kf_counters* counters, kf_diagnosis* out);

typedef struct kf_tuning {
  int32_t raster_group; /* GEMM: consecutive tiles walk this many tile rows
                           column by column (1..64; default 4)               */
  int32_t xcd_remap;    /* GEMM, CONV3D: 1 = the workgroups of one XCD take a
                           contiguous range of tiles (default), 0 = the
                           hardware's round-robin order                      */
  int32_t wg_per_cu;    /* CONV3D: persistent workgroups per compute unit,
                           1 or 2 (default 2)                                */
  int32_t variant;      /* kernel shape.  CONV2D_3X3 in the tiled family
                           (cin 64, cout 128, W 128, even H): 1 (default)
                           = the tile on 8 waves (64 x 64 wave blocks, two
                           per SIMD), 0 = on 4 waves (128 x 64), 2 = the
                           general kernel; any other CONV2D_3X3 shape: 2
                           only (4 rows x 32 columns x 128 channels per
                           workgroup).  GEMM (bf16 / fp8): 0 (default) =
                           256x256 tiles, one workgroup per CU; 1 = 128x256
                           tiles, two persistent workgroups per CU (B in KN
                           layout only; raster_group and xcd_remap unused);
                           2 = the 256x256 kernel storing a bf16 output
                           through LDS, each store instruction writing two
                           whole 512-byte tile rows (variant 0 stores
                           8-byte pieces from registers; the same bits).
                           Other ops: 0                                      */
} kf_tuning;

/* The plan's launch fields.  None of them changes a result bit: they reorder
   independent tiles, resize a persistent grid, or split a tile differently
   among waves with every output's sum over k taken in the same order.  kf_set_tuning validates
   the values (KF_ERR_INVALID_ARG) and takes effect at the next call. */
kf_status kf_get_tuning(const kf_desc* desc, kf_tuning* out);
kf_status kf_set_tuning(kf_desc* desc, const kf_tuning* tuning);

#define KF_MAX_TUNE_CANDIDATES 32

typedef struct kf_tune_result {
  int32_t n;            /* candidates timed                                  */
  int32_t best;         /* index of the one kept                             */
  kf_tuning config[KF_MAX_TUNE_CANDIDATES];
  double seconds[KF_MAX_TUNE_CANDIDATES]; /* time of one kf_fused_op (median
                                             round)                          */
  double panel_bytes[KF_MAX_TUNE_CANDIDATES]; /* GEMM: operand bytes the
                           candidate's tile order makes the eight L2s fetch
                           (model: per XCD and round of concurrently
                           resident tiles, one A panel per distinct tile row
                           and one B panel per distinct tile column); -1
                           for other plans                                   */
} kf_tune_result;

/* Time every candidate launch configuration of the plan on the caller's
   tensors -- in three interleaved rounds, each candidate once per round: one
   warm-up call, then `reps` (1..1000) calls between two HIP events on
   `stream` -- rank each by its median round (the clock drifts under power
   management), keep the fastest in the descriptor and report all of them in
   *result (seconds: the median round's mean time of one call).  Blocks
   until the stream is idle; outputs[0] holds the result of the last call
   (the same bits for every candidate).  Candidates: GEMM (bf16 / fp8) raster
   groups {1, 2, 4, 8, 16, 32, 64} x XCD order {contiguous, hardware} of the
   256x256 tile with each store path (variants 0 and 2), and the 128x256
   tile (variant 1) for B in KN layout; CONV3D
   workgroups per CU {2, 1} x XCD order; CONV2D_3X3 kernel variant {0, 1};
   every other plan has only its current configuration.  Kept: the fastest,
   except that among the GEMM candidates within 2% of the fastest time the
   one with the fewest panel_bytes is kept (the timing cannot tell such
   candidates apart; fewer L2 misses leave more HBM and fabric bandwidth to
   the epilogue). */
kf_status kf_autotune(kf_desc* desc, const kf_tensor* inputs, kf_tensor* outputs, void* stream, int32_t reps,
                      kf_tune_result* result);

/* ---- An entry point that allocates nothing ------------------------------
   For callers that cannot allocate device memory: code under HIP graph
   capture, tight serving loops, harnesses that forbid allocation.  Plans
   `spec` on the stack (no descriptor, no host or device allocation) and runs
   the fused operation exactly as kf_create + kf_fused_op would, with the
   library's static device scratch (4 MiB per GPU, held from the first call
   on a device until the process ends) in place of a descriptor workspace.
   Arguments, tensor rules and errors are those of kf_create and
   kf_fused_op; an op whose workspace exceeds the scratch (e.g. a row softmax
   with more than 512 K (row, 256-column tile) pairs) is rejected with
   KF_ERR_UNSUPPORTED before any device call, and so is a Conv3d chain that
   runs partly fused (it needs intermediate buffers).  Every call on one GPU uses the
   same scratch and nothing in it needs to start at zero (each call writes
   what it reads); calls that overlap on one GPU -- on different streams or
   host threads -- race on it and must be serialised by the caller.  Conv
   weights are repacked on every call. */
kf_status kf_fused_op_noalloc(const kf_op_spec* spec, const kf_tensor* inputs,
                              kf_tensor* outputs, void* stream);

/* A measured ceiling for the roofline beside the datasheet's: the matrix
   cores' sustained rate with no memory traffic.  One workgroup of 4 waves
   per compute unit, each SIMD issuing `iters` (1 .. 2^24) rounds of 8
   independent 32x32 MFMAs of `in_dtype` from registers (KF_BF16:
   v_mfma_f32_32x32x16_bf16; KF_FP8_E4M3: the 32x32x64 fp8 MFMA), after an
   untimed launch a tenth as long.  The datasheet's dense peaks assume the
   2.4 GHz peak engine clock; under sustained matrix-core load the clock is
   set by power management, and the probe reports it: every workgroup reads
   the shader-clock counter and the constant-rate counter at its start and
   end.  The roofline evaluation the paper's diagnosis rests on
   (Methodology, Diagnosis) compares a kernel with its hardware ceiling;
   this is that ceiling as the chip sustains it.  Allocates and frees a
   small device buffer and its own stream, and blocks until done.  Errors:
   KF_ERR_NO_DEVICE without a GPU, KF_ERR_UNSUPPORTED for other dtypes,
   KF_ERR_INVALID_ARG, KF_ERR_HIP. */
typedef struct kf_mfma_probe {
  double tflops;      /* FLOPs of the timed launch / its duration / 1e12     */
  double seconds;     /* the timed launch's duration (HIP events)            */
  double clock_ghz;   /* median over workgroups of shader-clock ticks per
                         second of constant-rate time, / 1e9                 */
  int32_t workgroups; /* launched (the device's compute units)               */
  int32_t reserved;   /* 0                                                   */
} kf_mfma_probe;

kf_status kf_probe_mfma(int32_t in_dtype, int64_t iters, kf_mfma_probe* out);

/* The memory side's measured ceiling: a plain device copy of `bytes` (a
   multiple of 16, at most 2^34) between two buffers this call allocates,
   16-byte loads and streaming stores over a grid-stride launch, one untimed
   copy then `reps` (1..1000) timed back to back.  A copy moves each byte
   twice (read and write); gbps counts both.  Allocates and frees 2 x bytes
   of device memory and its own stream, and blocks until done.  Errors:
   KF_ERR_NO_DEVICE, KF_ERR_INVALID_ARG, KF_ERR_OOM, KF_ERR_HIP. */
typedef struct kf_copy_probe {
  double gbps;        /* 2 x bytes / seconds / 1e9                           */
  double seconds;     /* one copy: the timed launches' total / reps          */
} kf_copy_probe;

kf_status kf_probe_copy(int64_t bytes, int32_t reps, kf_copy_probe* out);

/* Static description of a status code. */
const char* kf_status_string(kf_status status);

/* Thread-local message for the last failing call on this thread ("" if none). */
const char* kf_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* KF_H_ */
