// Internal declarations shared by the selector, the dispatcher and the kernels.
#pragma once

#include <cstddef>
#include <cstdint>

#include "../../include/conv_fwd.h"

namespace convfwd {

// Problem extents of Eq. (1); P, Q are the output extents.
struct Shape {
  int N, C, K, H, W, R, S;
  int P() const { return H - R + 1; }
  int Q() const { return W - S + 1; }
};

// Kernel families.
enum {
  FAMILY_STAGED = 1,  // global -> VGPR -> LDS staging, double buffered (any size)
  FAMILY_DMA = 2,     // global -> LDS direct buffer loads, NS-stage pipeline
  FAMILY_BF16 = 3,    // bf16 inputs: persistent, channel-fastest transposed LDS tiles
  FAMILY_STREAM1X1 = 4,  // pointwise: Ker resident in LDS, In streamed to registers (unrolled C)
  FAMILY_STREAM1X1_LOOP = 5,  // the same for any C % 4 == 0, looped over channel quads
  FAMILY_BF16_TR = 6,  // bf16 inputs, C = 32: shifted pixel-fastest LDS copies, transposing reads
  FAMILY_STREAM1X1_BAL = 7,  // pointwise, equal pixel share per workgroup: 32-pixel blocks in turn + k-split tail
};

// One compiled kernel instance (template parameters of the kernel family).
struct Variant {
  int id;
  int dtype;      // CONV_DTYPE_*
  int family;     // FAMILY_*
  int wk;         // 16-wide k blocks per wave (register tile along k)
  int wp;         // 16-wide pixel blocks per wave (register tile along pixels; for the
                  // unrolled streaming kernel in 16-pixel units: 2 * NB32 + NS16)
  int tc;         // input channels per pipeline step
  int rc, sc;     // compile-time R, S (0 = runtime)
  int max_ni;     // STAGED: max In staging elements per thread; DMA: In loads per wave per step;
                  // STREAM: 32-pixel blocks (unrolled) / phase-one 16-pixel blocks (looped)
  int max_nk;     // STAGED: max Ker staging vectors per thread; DMA: Ker loads per wave per step;
                  // STREAM: 16-pixel blocks (unrolled, 0 or 1) / phase-two blocks (looped)
  int ker_vec;    // Ker load width in elements
  int in_vec;     // In load width in elements (DMA family; 1 for STAGED)
  int threads;    // threads per workgroup
  int stages;     // pipeline depth (LDS buffers)
  int mfma32;     // DMA: 1 = 32x32x2 inner loop (64-row k tile, 32-pixel blocks)
  int nwc;        // DMA: groups of waves splitting each step's channels (0 = 1, no split)
  int phase_skip; // DMA: skips the zero taps of a stride-2 odd-tap layer's phases; runs only
                  // through conv_fwd_ex, reading In through the phase mapping
  int groups() const { return nwc > 1 ? nwc : 1; }
};

// Division by a divisor d >= 1 fixed for a launch, for numerators
// 0 <= n < 2^31: with s = ceil(log2 d) and m = ceil(2^(31+s) / d) (below
// 2^32), n / d = (n * m) >> (31 + s) exactly (the rounding error of m adds
// less than 1/d to n/d).  A 64-bit multiply and a shift in place of a
// 32-bit division (about 35 instructions per lane).  m = 0 marks a divisor
// the launch never divides by.
struct FastDiv {
  unsigned m;
  int s;
};

// Fully resolved launch geometry, passed by value to the kernels.
struct Geom {
  int N, C, K, H, W, R, S, P, Q;
  int tr, tw;                            // workgroup tile: output rows (flattened n*P+h) x cols
  int tiles_rows, tiles_cols, tiles_k;   // grid decomposition
  int in_rows, in_wp, in_cstride;        // LDS In tile: rows, row pitch, per-channel stride
  int ker_rstride;                       // LDS Ker tile: elements per k row
  int nwk, nwp;                          // waves along k and along pixels
  int order;                             // 0: k tiles innermost, 1: pixel tiles innermost
  int num_tiles;                         // workgroups
  int lds_in_elems, lds_ker_elems;       // LDS elements per pipeline buffer
  int ni_in, ni_ker;                     // staging loads per thread (In elements, Ker vectors)
  int nchunks;                           // pipeline steps = ceil(C / tc)
  unsigned in_bytes, ker_bytes;          // tensor sizes (DMA family range checks)
  int stage_elems, in_region;            // DMA family: LDS elements per stage / In part
                                         // (bf16 family: stage_elems = LDS bytes)
  int grid;                              // workgroups launched
  int split, cps;                        // channel ranges of the reduction; pipeline steps per range
  // Direct polyphase addressing (direct-to-LDS kernel, strided or padded
  // layers): In is the caller's tensor of C0 x H0 x W0 per image; inner
  // channel c' = (c * na + a) * nb + b at inner pixel (y', x') reads
  // In[c][sh * y' + a - ph][sw * x' + b - pw], zero outside the image.
  // nph = na * nb, or 0 when In is the inner tensor itself.  Wi: inner row
  // width when a 1x1 problem runs in its kernel view (one row of H' x W'
  // pixels per image), else 0.
  int nph, na, nb, sh, sw, ph, pw, C0, H0, W0, Wi;
  // The kernels' per-lane index maps divide by these (set_fast_divisors).
  FastDiv dv_in_cstride, dv_in_wp, dv_H, dv_ker_rstride, dv_tw, dv_P, dv_nph, dv_nb, dv_Wi, dv_tiles_k,
      dv_tiles_cols, dv_tiles_rows;
};

// Fills the FastDiv fields of g from its extents (after every other field).
void set_fast_divisors(Geom* g);

const Variant* variants(int* count);
const Variant* find_variant(int id);

// Resolve a plan's tile fields into a launch geometry; false if infeasible.
bool resolve_geom(const Shape& s, const Variant& v, const conv_plan_t& plan, Geom* g, int* lds_bytes);

// Launch the kernel of variant v (asynchronous).  Returns a conv_status_t.
int launch(const Variant& v, const Geom& g, const void* In, const void* Ker, float* Out, void* stream);
// Launch of a bf16-input plan writing bf16 Out (round to nearest even): the
// transposing bf16 kernel writes it directly; other kernels write fp32 to a
// stream-ordered workspace that a second kernel rounds into Out.
int launch_bf16_out(const Variant& v, const Geom& g, const void* In, const void* Ker, void* Out, void* stream);
// Exact bf16 -> fp32 widening, and fp32 -> bf16 rounding (nearest even), of
// n elements on `stream`.
int launch_widen_bf16(const void* src, float* dst, int64_t n, void* stream);
int launch_round_bf16(const float* src, void* dst, int64_t n, void* stream);

// Polyphase rewrite of a strided, padded convolution into a stride-1 valid
// one (conv_fwd_ex): na x nb phases per input channel, inner extents
// Hp x Wp and taps Rp x Sp.
struct PhaseGeom {
  int N, C, K, H, W, R, S;
  int sh, sw, ph, pw;
  int na, nb;  // phases along rows / columns: min(sh, R), min(sw, S)
  int Hp, Wp;  // inner input extents: P + Rp - 1, Q + Sp - 1
  int Rp, Sp;  // inner taps: ceil(R / sh), ceil(S / sw)
  int P, Q;    // output extents
};
// Geometry g of an inner plan (variant v) rewritten to read the caller's In
// of the strided, padded problem p through the phase mapping; false when the
// kernel cannot (not the direct-to-LDS family, vector In loads, a pipeline
// step that splits a channel's phases, or In of 2 GB or more).
bool phase_direct(const Variant& v, const PhaseGeom& p, int dtype, Geom* g);
// Stream-ordered device memory from the library's per-device pool
// (hipMallocFromPoolAsync / hipFreeAsync on `stream`).
int stream_alloc(size_t bytes, void* stream, void** out);
int stream_free(void* p, void* stream);
// A call's workspace: the buffer the library keeps for (current device,
// stream, nesting level) -- levels 0 (conv_fwd_ex, bf16 widening), 1 (bf16
// Out staging), 2 (split partial sums) let nested steps of one call hold
// theirs together -- or, while another host thread holds that buffer, a
// fresh stream-ordered allocation.  Release enqueues nothing for a kept
// buffer: the next call on the stream reuses it in stream order.
struct Workspace {
  void* ptr = nullptr;
  bool cached = false;
  bool arena = false;  // carved from the calling thread's ScratchArena
  int level = 0;
};
int workspace_acquire(int level, size_t bytes, void* stream, Workspace* w);
int workspace_release(const Workspace& w, void* stream);
// Frees (stream-ordered) the buffers kept for `stream` on the current device.
int workspace_release_stream(void* stream);
// Allocation-free calls: while an arena is installed on the calling thread,
// workspace_acquire carves every workspace from it (bump allocation,
// 256-byte aligned; CONV_ESCRATCH when it is full) and release is a no-op.
struct ScratchArena {
  char* base;
  size_t cap;
  size_t used;
};
void set_thread_arena(ScratchArena* a);
// Device address of the current device's copy of the library's static
// scratch array (CONV_NOALLOC_SCRATCH_BYTES), looked up once per device.
int noalloc_scratch(void** base);
// Phase-split In into Inp (Inp non-null) and Ker into Kp (Kp non-null), on
// `stream`.
int launch_phase_split(const PhaseGeom& p, int dtype, const void* In, const void* Ker, void* Inp, void* Kp,
                       void* stream);
// Median duration in microseconds of `reps` launches on `stream` after one
// untimed launch, each between its own two HIP events and preceded by a pass
// over a 512 MB stream-ordered scratch buffer (cold caches); waits for the
// stream.
int time_launches(const Variant& v, const Geom& g, const void* In, const void* Ker, float* Out,
                  void* stream, int reps, float* us);

// Selector entry points (host only, no HIP calls).
int select_plan(const Shape& s, int dtype, conv_plan_t* out);
// phase_skip: also the phase-skip variants (conv_fwd_ex's stride-2 odd-tap
// layers, read through the phase mapping; they are wrong for any other use)
int enumerate_plans(const Shape& s, int dtype, conv_plan_t* plans, int cap, bool phase_skip = false);
int score_plan(const Shape& s, conv_plan_t* plan);  // fills the derived fields of a plan

// Paper model, Sec. 3.2: per-array volumes for a permutation (codes n=0..w=6).
void model_volume(const int perm[7], const int64_t N[7], const int64_t T[7], int out_factor,
                  double dv[3]);

}  // namespace convfwd
