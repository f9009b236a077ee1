/*
 * conv_fwd.h -- C ABI of the MI355X (gfx950) forward-convolution library.
 *
 * The operation (Sec. 1, Eq. (1); loop bounds of Listing 2):
 *
 *   Out[n][k][h][w] = sum_{c<C, r<R, s<S} In[n][c][h+r][w+s] * Ker[k][c][r][s]
 *
 * for n < N, k < K, h < P = H-R+1, w < Q = W-S+1.  H and W are the *input*
 * height and width (caption of Table 1); the correlation is valid (no
 * padding), stride 1, with no kernel flip.  Out is overwritten (beta = 0).
 *
 * Layouts (Sec. 9, artifact appendix): In is NCHW, Ker is KCRS, Out is NKPQ;
 * all dense, contiguous, row-major.  Only element alignment is required: the
 * selected kernel depends on the shape and on whether In and Ker are 16-byte
 * aligned (kernels with vector loads need it).
 *
 * Loop order and tile sizes are chosen per shape by a tile selector built on
 * the paper's data-movement model (Sec. 3-5, Algorithm 1 of Sec. 8),
 * re-derived for the gfx950 memory hierarchy; see conv_fwd_plan.
 *
 * Ownership: every tensor pointer is DEVICE memory allocated and freed by
 * the caller.  The library keeps a host-side plan cache; its device
 * allocations are workspaces (split reductions, the strided rewrite, bf16
 * fallbacks, conv_fwd_tune's scratch) from a memory pool the library
 * creates per device, which keeps up to 1 GB of freed blocks for reuse.
 * The workspaces of the compute calls are kept per device, stream and
 * nesting level and reused by the next call on that stream (stream order
 * makes that safe); each grows to the largest size a call on that stream
 * needed and is held until conv_fwd_release_workspaces(stream) frees it or
 * the process ends.  Call conv_fwd_release_workspaces before destroying a
 * stream: a buffer kept for a destroyed stream stays held, and a new stream
 * that gets the same handle value would reuse it in its own stream order,
 * which is safe only once the old stream's work has finished.  A call that
 * finds its buffer held by another host thread takes and returns a fresh one
 * in stream order.  conv_fwd_ex_noalloc allocates nothing (see there).
 * The calling thread's current device must own the stream.
 * In, Ker and Out must not overlap.
 *
 * Asynchrony: the compute calls enqueue kernels on `stream` (a hipStream_t;
 * NULL = the default stream) and return without synchronising.  A return of
 * CONV_OK means the launch was enqueued; faults inside the kernel surface at
 * the caller's next synchronisation.
 *
 * Errors: argument and plan validation errors (CONV_EINVAL, CONV_ENULL,
 * CONV_ERANGE, CONV_ENOPLAN, CONV_ESCRATCH) are reported before anything is
 * launched, and Out is untouched.  A call that runs several kernels (the
 * strided rewrite, bf16 widening or bf16 Out staging, split reductions) can
 * return CONV_EHIP after an earlier kernel of the call was enqueued; Out is
 * then unspecified.
 * Thread safety: all entry points are reentrant.
 */
#ifndef CONV_FWD_H
#define CONV_FWD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CONV_OK = 0,
  CONV_EINVAL = -1,  /* an extent <= 0, R > H, S > W, or a bad plan/option */
  CONV_ENULL = -2,   /* a null tensor or output-struct pointer */
  CONV_ERANGE = -3,  /* a tensor of 2^31 elements or more */
  CONV_ENOPLAN = -4, /* no kernel configuration fits the shape */
  CONV_EHIP = -5,    /* the HIP runtime reported an error at launch */
  CONV_ESCRATCH = -6 /* conv_fwd_ex_noalloc: the call needs more scratch than
                        CONV_NOALLOC_SCRATCH_BYTES */
} conv_status_t;

/* Element types of In and Ker (Out and accumulation are always fp32). */
enum { CONV_DTYPE_F32 = 0, CONV_DTYPE_BF16 = 1 };

/* Memory levels of the model, innermost first. */
enum {
  CONV_LVL_REG = 0,  /* LDS -> VGPR operand traffic of the wave tiles      */
  CONV_LVL_LDS = 1,  /* L2 -> LDS traffic of the workgroup tiles           */
  CONV_LVL_L2 = 2,   /* MALL/HBM -> L2 traffic of the per-XCD tile sets    */
  CONV_LVL_HBM = 3,  /* device-memory traffic (compulsory In, Ker, Out)    */
  CONV_NUM_LVLS = 4
};

/*
 * A tile plan: one point of the search space of Algorithm 1 (Sec. 8) for the
 * gfx950 kernel, with the model's prediction of its data movement.
 *
 * The workgroup (LDS-level) tile covers `tile_k` output channels and a block
 * of output pixels: `tile_rows` consecutive output rows of the flattened
 * (n, h) row index times `tile_cols` consecutive columns, with `tile_c` input
 * channels staged per pipeline step (all R x S taps at once).  The wave
 * (register-level) tile is `wave_k` x `wave_px`; accumulators stay in
 * registers for the whole reduction (the Out-stationary classes
 * <{n,k,h,w},{c,r},s> / <{n,k,h,w},{c,s},r> of Sec. 4).  Exception: the
 * balanced pointwise kernel of 1x1 layers takes `tile_cols` pixels of the
 * flattened n*H*W index per workgroup, not as one range but as 128-pixel
 * blocks handed out in grid stride plus one 16-pixel tail block.
 */
typedef struct {
  int dtype;          /* CONV_DTYPE_*                                        */
  int variant;        /* internal kernel variant id (opaque)                 */
  int tile_k;         /* output channels per workgroup                      */
  int tile_rows;      /* output rows (flattened n*P+h) per workgroup         */
  int tile_cols;      /* output columns per workgroup                        */
  int tile_c;         /* input channels per pipeline step                    */
  int wave_k;         /* output channels per wave                            */
  int wave_px;        /* output pixels per wave (multiple of 16)             */
  int waves_k;        /* waves along k in a workgroup                        */
  int waves_px;       /* waves along pixels in a workgroup                   */
  int grid_order;     /* 0: k tiles innermost in the workgroup order (In reuse
                         in L2); 1: pixel tiles innermost (Ker reuse)        */
  int split_c;        /* input-channel ranges the reduction is split into
                         (0 or 1 = none).  Above 1 (direct-to-LDS plans only),
                         each range's partial Out goes to a stream-ordered
                         temporary workspace of split_c x |Out| floats
                         (the library's pool, on the call's stream) and a
                         second kernel adds the ranges in fixed order, so
                         results stay deterministic.                       */
  int reserved;       /* 0                                                   */
  int lds_bytes;      /* dynamic LDS per workgroup                           */
  int64_t num_wg;     /* workgroups launched                                 */
  int class_lvl[CONV_NUM_LVLS]; /* paper class 1..8 (Sec. 4) per level, 0 = n/a */
  double pred_bytes[CONV_NUM_LVLS]; /* modelled bytes moved at each level    */
  double pred_us[CONV_NUM_LVLS];    /* bytes / bandwidth of each level, us   */
  double pred_mfma_us;              /* MFMA time incl. padding and waves, us */
  double pred_total_us;             /* max over the above (Sec. 5 min-max)
                                       plus the pipeline's fill and drain     */
  double rank_us;                   /* pred_total_us times the kernel family's
                                       measured factor: the selector's order  */
  double paper_bytes[CONV_NUM_LVLS]; /* the paper's Sec. 3.2 volume of the
                                       level's permutation class and tile, in
                                       bytes, before line rounding (0 = the
                                       level has no such form)               */
} conv_plan_t;

/*
 * fp32 forward convolution, Eq. (1).
 *   In  : [N][C][H][W]           fp32, device
 *   Ker : [K][C][R][S]           fp32, device
 *   Out : [N][K][H-R+1][W-S+1]   fp32, device, overwritten
 * Returns a conv_status_t.
 */
int conv_fwd(int N, int C, int K, int H, int W, int R, int S,
             const float* In, const float* Ker, float* Out, void* stream);

/*
 * bf16-input forward convolution, Eq. (1): In and Ker hold bfloat16 bit
 * patterns (uint16, same layouts as above); products and sums are formed in
 * fp32 and Out is fp32.  Returns a conv_status_t.
 */
int conv_fwd_bf16(int N, int C, int K, int H, int W, int R, int S,
                  const uint16_t* In, const uint16_t* Ker, float* Out, void* stream);

/*
 * bf16-input forward convolution with bf16 output: as conv_fwd_bf16 (fp32
 * products and sums), then each output rounded to the nearest bf16 (ties to
 * even), halving the bytes written.  Out : [N][K][H-R+1][W-S+1] bf16 bit
 * patterns, device.  The plan is the one conv_fwd_bf16 selects, except
 * where that plan's transposing-read kernel could not pair its stores into
 * 16-byte pieces although Out allows them (16-byte aligned Out and
 * (W-S+1) % 8 == 0): then the best candidate that pairs them
 * (conv_fwd_bf16_out_plan).  The transposing-read bf16 kernel writes bf16
 * directly, any other kernel writes fp32 into a stream-ordered workspace
 * (from the library's pool, returned within the call) that a second kernel
 * rounds into Out.
 * The paper states single precision only; the other entry points write
 * fp32 Out, and this one is the bf16-output refinement that makes bf16
 * layers less write-bound.  Returns a conv_status_t.
 */
int conv_fwd_bf16_out(int N, int C, int K, int H, int W, int R, int S,
                      const uint16_t* In, const uint16_t* Ker, uint16_t* Out, void* stream);

/*
 * Strided, zero-padded forward convolution.  The paper presents Eq. (1)
 * without stride and notes that the method carries over (Sec. 3.1,
 * footnote 1); Table 1 includes stride-2 layers.  The operation:
 *
 *   Out[n][k][h][w] = sum_{c<C, r<R, s<S} X[n][c][h*sh + r - ph][w*sw + s - pw] * Ker[k][c][r][s]
 *
 * with X = In inside [0,H) x [0,W) and zero outside, for
 * h < P = (H + 2 ph - R) / sh + 1 and w < Q = (W + 2 pw - S) / sw + 1.
 *   stride_h, stride_w : 1 .. 64;  pad_h, pad_w : 0 .. 4096 (zeros each side)
 *   dtype : CONV_DTYPE_*; In/Ker fp32 or bf16 bit patterns as for conv_fwd
 *           and conv_fwd_bf16 (same layouts); Out [N][K][P][Q] fp32
 * Stride 1 without padding is conv_fwd / conv_fwd_bf16.  Otherwise the call
 * rewrites the problem as a stride-1 valid convolution (each input channel
 * becomes min(sh,R) x min(sw,S) phase images; Ker gets ceil(R/sh) x
 * ceil(S/sw) taps, zero where no original tap lands) and runs the selected
 * stride-1 plan of the inner problem (see conv_fwd_ex_inner_shape and
 * conv_fwd_ex_plan).  For fp32 plans on the direct-to-LDS kernel (and on
 * the balanced pointwise kernel for 1x1 layers) the kernel reads In through
 * the phase mapping (see conv_fwd_ex_geometry); otherwise a small kernel
 * writes the phase images into a workspace first.  For stride-2 layers with
 * odd taps (R = 2 ceil(R/2) - 1, likewise S) the plan may be a phase-skip
 * variant of the direct-to-LDS kernel, which leaves out the zero taps of the
 * phases (3x3: 7 of 16).  With more
 * than one phase per channel, another small kernel writes the rearranged
 * Ker into a workspace.  Workspaces are the per-stream ones described under
 * Ownership.  Asynchronous like conv_fwd.  Returns a conv_status_t.
 */
int conv_fwd_ex(int N, int C, int K, int H, int W, int R, int S,
                int stride_h, int stride_w, int pad_h, int pad_w, int dtype,
                const void* In, const void* Ker, float* Out, void* stream);

/*
 * Allocation-free variant of conv_fwd_ex, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, layouts, operation and
 * results as conv_fwd_ex (the same plans and kernels run), but every
 * workspace the call needs (phase images of In, the rearranged Ker, split
 * partial sums, bf16 widening) is carved from one static device array of
 * CONV_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends; the call makes no hipMalloc, hipFree or other
 * allocating call.  A call that would need more scratch returns
 * CONV_ESCRATCH before launching anything.  Every call on one GPU shares
 * that GPU's array (which keeps the previous call's contents, and nothing
 * in it is assumed zero): calls that overlap on one GPU -- on different
 * streams, or from different host threads -- race and must be serialised
 * by the caller.  Returns a conv_status_t.
 */
#define CONV_NOALLOC_SCRATCH_BYTES (64 * 1024 * 1024)
int conv_fwd_ex_noalloc(int N, int C, int K, int H, int W, int R, int S,
                        int stride_h, int stride_w, int pad_h, int pad_w, int dtype,
                        const void* In, const void* Ker, float* Out, void* stream);

/*
 * Host-only: the plan conv_fwd_bf16_out runs for this shape with a 16-byte
 * aligned Out (see there).  Makes no HIP call.  Returns a conv_status_t;
 * CONV_ENOPLAN where no bf16 kernel instance takes the shape (the call then
 * widens the inputs and runs the fp32 plan).
 */
int conv_fwd_bf16_out_plan(int N, int C, int K, int H, int W, int R, int S, conv_plan_t* plan_out);

/*
 * Host-only: the inner stride-1 problem conv_fwd_ex runs for these
 * arguments, as inner[0..8] = N, C', K, H', W', R', S' (the shape to pass to
 * conv_fwd_plan / conv_fwd_candidates) followed by the output extents P, Q.
 * Returns a conv_status_t.
 */
int conv_fwd_ex_inner_shape(int N, int C, int K, int H, int W, int R, int S,
                            int stride_h, int stride_w, int pad_h, int pad_w, int32_t inner[9]);

/*
 * Host-only: the tile plan the selector picks for this shape and dtype
 * (CONV_DTYPE_*), with its modelled per-level bytes.  Cached per shape.
 * Makes no HIP call.  Returns a conv_status_t.
 */
int conv_fwd_plan(int N, int C, int K, int H, int W, int R, int S, int dtype,
                  conv_plan_t* plan_out);

/*
 * Forward convolution with an explicit plan (as returned by conv_fwd_plan,
 * possibly with other tile fields, e.g. for model-validation sweeps).  The
 * plan is re-validated: only its dtype, variant, tile_* , wave_*, waves_*,
 * grid_order and split_c fields are read; the rest is recomputed.  A split_c
 * above 1 runs the split reduction with its workspace of split_c x |Out|
 * floats.  `In`/`Ker` are fp32
 * or bf16 per plan->dtype.  Returns CONV_EINVAL for a plan the kernels cannot
 * run -- including a plan whose vector loads need 16-byte aligned In or Ker
 * when the tensors passed are not, and a phase-skip plan (conv_fwd_ex
 * only) -- else as conv_fwd.
 */
int conv_fwd_with_plan(int N, int C, int K, int H, int W, int R, int S,
                       const void* In, const void* Ker, float* Out,
                       const conv_plan_t* plan, void* stream);

/*
 * Host-only: scores a plan's tile fields for this shape, as the selector
 * does for its candidates.  Reads dtype, variant, tile_*, wave_*, waves_*,
 * grid_order and split_c; writes every derived field (lds_bytes, num_wg,
 * class_lvl, pred_*, rank_us, paper_bytes).  Returns CONV_OK, or CONV_EINVAL
 * for a plan the kernels cannot run (the plan is then unchanged).  Makes no
 * HIP call.
 */
int conv_fwd_score_plan(int N, int C, int K, int H, int W, int R, int S, conv_plan_t* plan);

/*
 * Host-only: every candidate plan the selector scores for this shape (the
 * feasible kernel configurations), best first.  Writes at most `cap` plans
 * to `plans` (may be NULL when cap == 0) and returns the number of
 * candidates, or a negative conv_status_t.
 */
int conv_fwd_candidates(int N, int C, int K, int H, int W, int R, int S, int dtype,
                        conv_plan_t* plans, int cap);

/*
 * Limited empirical tuning over the model's best plans (the MOpt-5 variant
 * of Sec. 10: the model ranks the configurations, the top few are run and
 * the fastest is kept, which sidesteps effects the model does not capture).
 *
 * Times the first `top_n` candidates of conv_fwd_candidates (best first)
 * that run with these tensors' alignment: each gets one untimed launch and
 * then `reps` launches on `stream`, each between its own two HIP events and
 * after a read pass over a 512 MB scratch buffer, so that the caches hold
 * none of In (as when each call of a network brings new data); the median
 * launch time in microseconds goes to times_us[i] (times_us may be NULL;
 * else room for top_n floats).  The scratch buffer is taken from and
 * returned to the library's memory pool in stream order.  The fastest plan
 * is written to *plan_out and becomes the cached plan of this shape, dtype
 * and tensor alignment: later
 * conv_fwd / conv_fwd_bf16 / conv_fwd_plan calls for them return or run it.
 *   dtype      : CONV_DTYPE_*; In and Ker as for conv_fwd or conv_fwd_bf16
 *   Out        : overwritten with Eq. (1) (every candidate computes it)
 *   top_n      : 1 .. CONV_TUNE_MAX;  reps : 1 .. 1000
 * Unlike the other compute calls this one blocks until the stream has run
 * the timed launches (it waits on the second event of each candidate).
 * Returns the number of plans timed (>= 1), or a negative conv_status_t; on
 * an error after the first launch Out may hold a partial result and the
 * cache is unchanged.
 */
#define CONV_TUNE_MAX 64
int conv_fwd_tune(int N, int C, int K, int H, int W, int R, int S, int dtype,
                  const void* In, const void* Ker, float* Out, int top_n, int reps,
                  void* stream, conv_plan_t* plan_out, float* times_us);

/*
 * Host-only: the paper's single-level data-movement volume (Sec. 3.2) for a
 * tile-loop permutation.  perm[0..6] lists the loops outermost first, coded
 * n=0, k=1, c=2, r=3, s=4, h=5, w=6; N[] and T[] are problem extents and
 * tile sizes in the same coding (h, w extents are output extents).  Writes
 * the In, Ker and Out volumes in elements to dv[0..2], Out multiplied by
 * out_factor (2 in the paper: read and write).  Returns a conv_status_t.
 */
int conv_model_volume(const int perm[7], const int64_t N[7], const int64_t T[7],
                      int out_factor, double dv[3]);

/*
 * Host-only introspection: the launch geometry a plan resolves to for this
 * shape, as CONV_GEOM_FIELDS int32 values in this order:
 *   kernel view of the problem N, C, K, H, W, R, S, P, Q (a 1x1 problem is
 *   presented as one row of H*W pixels per image);
 *   tile rows, tile cols; row tiles, column tiles, k tiles;
 *   LDS In rows, In row pitch, In channel stride; LDS Ker row pitch;
 *   waves along k, waves along pixels; grid order; workgroups;
 *   LDS In / Ker elements per buffer; staging loads per thread (In, Ker);
 *   pipeline steps; then the kernel variant's k blocks per wave, pixel blocks
 *   per wave, channels per step, compile-time R, S (0 = runtime), staging
 *   capacity (In, Ker), Ker vector width, threads per workgroup; LDS bytes;
 *   kernel family (1 register-staged, 2 direct-to-LDS, 3 bf16, 4 / 5
 *   pointwise streaming unrolled / looped), In vector
 *   width, pipeline stages, LDS elements per stage (family 3: LDS bytes), In
 *   elements per stage (family 2), In and Ker bytes, workgroups launched;
 *   1 if the kernel skips the zero taps of a stride-2 odd-tap layer's phases
 *   (family 2; such plans run only through conv_fwd_ex, and
 *   conv_fwd_geometry rejects them), then two reserved zeros; channel ranges
 *   of the reduction, pipeline steps
 *   per range; 1 if the inner loop is on 32x32x2 MFMAs (family 2); groups
 *   of waves that split each pipeline step's channels inside the workgroup
 *   (family 2; 1 otherwise); then the direct phase addressing of
 *   conv_fwd_ex_geometry (all zero here): phases per input channel
 *   (0 = none), phases along rows and columns, stride (rows, columns),
 *   padding (rows, columns), the caller's In channels, height and width,
 *   and the inner row width of a 1x1 problem run as one row of pixels per
 *   image (0 otherwise); then, for the divisors the kernels' index maps use
 *   (In channel stride, In row pitch, H, Ker row pitch, tile columns, P,
 *   phases per channel, phases along columns, the 1x1 inner row width, k
 *   tiles, column tiles, row tiles), the pair (m as a uint32 bit pattern, s)
 *   with which the kernels compute n / d as (n * m) >> (31 + s) for
 *   0 <= n < 2^31 (m = 0: not divided by).
 * Writes min(cap, CONV_GEOM_FIELDS) values and returns CONV_GEOM_FIELDS, or
 * a negative conv_status_t (CONV_EINVAL for a plan the kernels cannot run).
 */
#define CONV_GEOM_FIELDS 87
int conv_fwd_geometry(int N, int C, int K, int H, int W, int R, int S,
                      const conv_plan_t* plan, int32_t* out, int cap);

/*
 * Host only: the launch geometry conv_fwd_ex uses for `plan`, a plan of its
 * inner stride-1 problem (conv_fwd_ex_inner_shape).  The layout is that of
 * conv_fwd_geometry.  When the plan's kernel reads the caller's In directly
 * through the phase mapping (fp32, the direct-to-LDS family with scalar In
 * loads and whole channels per pipeline step, In below 2 GB), the last
 * eleven fields describe that mapping: inner channel c' = (c * na + a) * nb + b at
 * inner pixel (y', x') reads In[c][sh * y' + a - ph][sw * x' + b - pw], zero
 * outside the image (Sec. 3 defines the loop nest; stride and padding are
 * the rewrite of conv_fwd_ex).  Otherwise those fields are zero and
 * conv_fwd_ex phase-splits In into a workspace first.  Returns
 * CONV_GEOM_FIELDS or a negative conv_status_t.
 */
int conv_fwd_ex_geometry(int N, int C, int K, int H, int W, int R, int S, int stride_h, int stride_w,
                         int pad_h, int pad_w, const conv_plan_t* plan, int32_t* out, int cap);

/*
 * Host only: the plan conv_fwd_ex runs for this layer with 16-byte aligned
 * tensors -- the selector's plan of its inner stride-1 problem.  *direct (if
 * non-null) is set to 1 when that plan's kernel reads the caller's In
 * through the phase mapping (fp32 layers with stride or padding, see
 * conv_fwd_ex_geometry), else 0 (In is phase-split into a workspace first,
 * or the layer needs no rewrite).  Returns CONV_OK or a negative
 * conv_status_t.
 */
int conv_fwd_ex_plan(int N, int C, int K, int H, int W, int R, int S, int stride_h, int stride_w, int pad_h,
                     int pad_w, int dtype, conv_plan_t* plan_out, int32_t* direct);

/*
 * Frees, in the order of `stream` (hipFreeAsync), the workspaces the compute
 * calls keep for that stream on the calling thread's current device (see
 * Ownership).  Call it before destroying a stream the library has used; a
 * later call on the stream takes a new workspace.  Returns a conv_status_t.
 */
int conv_fwd_release_workspaces(void* stream);

/* Static string for a conv_status_t. */
const char* conv_fwd_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* CONV_FWD_H */
