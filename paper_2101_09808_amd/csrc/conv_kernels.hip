// Forward convolution kernels for gfx950 (CDNA4), Eq. (1):
//   Out[n][k][h][w] = sum_{c,r,s} In[n][c][h+r][w+s] * Ker[k][c][r][s]
//
// Structure (one workgroup = one tile of the non-reduction loops, Sec. 7):
//   * The grid enumerates workgroup tiles of (k, pixel) -- pixels are a range
//     of rows of the flattened (n, h) output-row index times a range of
//     columns.  The linear order of the tiles is the outer tile-loop order
//     chosen by the selector (k tiles innermost or pixel tiles innermost), and
//     consecutive tiles of that order are mapped to the same XCD so that they
//     share its L2.
//   * Per pipeline step the workgroup stages `TC` input channels of the In
//     halo tile (rows h..h+tile+R-1, Eq. (4)'s (T_h + T_r - 1)(T_w + T_s - 1)
//     footprint) and the matching Ker tile [tile_k][TC*R*S] in LDS, double
//     buffered: the global loads of step i+1 are issued before the MFMAs of
//     step i.
//   * Each wave keeps a (16*WK) x (16*WP) tile of Out in accumulator
//     registers for the whole reduction (the Out-stationary classes of Sec. 4,
//     reduction loops c, r, s innermost) and issues one 16x16x4 fp32 MFMA per
//     (k block, pixel block, 4 channels, tap).  This plays the part of the
//     paper's outer-product microkernel (Sec. 6): an MFMA is an outer-product
//     accumulation done by the matrix core, and WK*WP independent
//     accumulators keep enough MFMAs in flight to cover their latency.
//   * Epilogue: each accumulator element is stored once; 16 consecutive lanes
//     hold 16 consecutive output pixels, so stores coalesce.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <tuple>
#include <type_traits>
#include <utility>
#include <vector>

#include "conv_internal.h"

namespace convfwd {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));

template <int N>
struct FVec {
  typedef float type __attribute__((ext_vector_type(N)));
};
template <>
struct FVec<1> {
  typedef float type;
};

constexpr int kThreads = 256;

// Hardware dispatches workgroup b to XCD b % 8.  Give XCD x the contiguous
// range [x*G8/8, (x+1)*G8/8) of the logical tile order (tail left as is).
__device__ __forceinline__ int xcd_remap(int b, int G) {
  const int G8 = G & ~7;
  return (b < G8) ? (b & 7) * (G8 >> 3) + (b >> 3) : b;
}

// n / d for 0 <= n < 2^31 with the launch's precomputed multiplier (FastDiv).
__device__ __forceinline__ int fdiv(int n, FastDiv f) {
  return (int)(((unsigned long long)(unsigned)n * f.m) >> (31 + f.s));
}

struct TileCoord {
  int rho0, rho_end;  // output rows [rho0, rho_end) of the flattened n*P+h index
  int q0, tw_eff;     // output columns [q0, q0 + tw_eff)
  int k0;             // first output channel
  int nu0, nrows;     // input rows [nu0, nu0 + nrows) of the flattened n*H+y index
};

// Output tile of workgroup b (0 <= b < num_tiles), in the grid order.
__device__ __forceinline__ TileCoord tile_coord(const Geom& g, int BK, int b) {
  const int L = xcd_remap(b, g.num_tiles);
  int kt, ct, rt;
  if (g.order == 0) {
    const int rest = fdiv(L, g.dv_tiles_k);
    kt = L - rest * g.tiles_k;
    rt = fdiv(rest, g.dv_tiles_cols);
    ct = rest - rt * g.tiles_cols;
  } else {
    const int rest = fdiv(L, g.dv_tiles_cols);
    ct = L - rest * g.tiles_cols;
    kt = fdiv(rest, g.dv_tiles_rows);
    rt = rest - kt * g.tiles_rows;
  }
  TileCoord t;
  const int NP = g.N * g.P;
  t.rho0 = rt * g.tr;
  t.rho_end = min(t.rho0 + g.tr, NP);
  t.q0 = ct * g.tw;
  t.tw_eff = min(g.tw, g.Q - t.q0);
  t.k0 = kt * BK;
  const int nf = fdiv(t.rho0, g.dv_P), pf = t.rho0 - nf * g.P;
  t.nu0 = nf * g.H + pf;
  const int nl = fdiv(t.rho_end - 1, g.dv_P), pl = (t.rho_end - 1) - nl * g.P;
  t.nrows = nl * g.H + pl + g.R - t.nu0;
  return t;
}

// ---------------------------------------------------------------------------
// fp32 kernel.  WK x WP blocks of 16x16 per wave, TC channels per step,
// compile-time taps RC x SC (0 = runtime), staging arrays of MAXNI In
// elements and MAXNK Ker vectors of KV floats per thread.
template <int WK, int WP, int TC, int RC, int SC, int MAXNI, int MAXNK, int KV>
__global__ void __launch_bounds__(kThreads)
conv_f32_kernel(const float* __restrict__ In, const float* __restrict__ Ker,
                float* __restrict__ Out, const Geom g) {
  typedef typename FVec<KV>::type kvec_t;
  extern __shared__ __align__(16) float lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int j = lane & 15, gq = lane >> 4;
  const int wk = wave % g.nwk, wp = wave / g.nwk;
  const int BK = 16 * WK * g.nwk;
  const int R = RC ? RC : g.R, S = SC ? SC : g.S;
  const int RS = R * S;
  const int H = g.H, W = g.W, C = g.C, K = g.K;
  const TileCoord t = tile_coord(g, BK, (int)blockIdx.x);

  // Per-thread staging list for the In halo tile: element idx = tid + 256*i
  // of the [TC][in_rows][in_wp] LDS image.  in_goff is the global offset
  // relative to channel c0 (-1: outside the tile, stage a zero); in_lc packs
  // the LDS offset (low 20 bits) and the channel within the step.
  int in_goff[MAXNI], in_lc[MAXNI];
  {
    const int E = g.in_rows * g.in_wp;
    const int ncols = t.tw_eff + S - 1;
#pragma unroll
    for (int i = 0; i < MAXNI; ++i) {
      const int idx = tid + kThreads * i;
      in_lc[i] = -1;
      in_goff[i] = -1;
      if (i < g.ni_in && idx < TC * E) {
        const int cl = idx / E, e = idx - cl * E;
        const int row = e / g.in_wp, x = e - row * g.in_wp;
        in_lc[i] = (cl * g.in_cstride + e) | (cl << 20);
        if (row < t.nrows && x < ncols) {
          const int nu = t.nu0 + row;
          const int n = nu / H, y = nu - n * H;
          in_goff[i] = ((n * C + cl) * H + y) * W + t.q0 + x;
        }
      }
    }
  }
  // Per-thread staging list for the Ker tile [BK][TC*RS] (row pitch
  // ker_rstride in LDS), in vectors of KV: packed (row << 16 | column), or -1.
  const int TCRS = TC * RS;
  int ker_km[MAXNK];
  {
    const int per_row = TCRS / KV;
#pragma unroll
    for (int i = 0; i < MAXNK; ++i) {
      const int idx = tid + kThreads * i;
      ker_km[i] = -1;
      if (i < g.ni_ker && idx < BK * per_row) {
        const int kl = idx / per_row, m = (idx - kl * per_row) * KV;
        ker_km[i] = (kl << 16) | m;
      }
    }
  }
  // Per-lane LDS offsets of this lane's output pixel in each pixel block.
  const int tpx = g.tr * g.tw;
  int poff[WP];
#pragma unroll
  for (int pb = 0; pb < WP; ++pb) {
    const int px = (wp * WP + pb) * 16 + j;
    const int row_i = px / g.tw, col = px - row_i * g.tw;
    const int rho = t.rho0 + row_i;
    int off = 0;  // masked pixels read a valid, zero-filled LDS location
    if (px < tpx && rho < t.rho_end && col < t.tw_eff) {
      const int n = rho / g.P, p = rho - n * g.P;
      off = (n * H + p - t.nu0) * g.in_wp + col;
    }
    poff[pb] = off;
  }
  int koff[WK];
#pragma unroll
  for (int kb = 0; kb < WK; ++kb) koff[kb] = ((wk * WK + kb) * 16 + j) * g.ker_rstride;

  v4f acc[WK][WP];
#pragma unroll
  for (int kb = 0; kb < WK; ++kb)
#pragma unroll
    for (int pb = 0; pb < WP; ++pb) acc[kb][pb] = v4f{0.f, 0.f, 0.f, 0.f};

  float in_st[MAXNI];
  kvec_t ker_st[MAXNK];
  const int kcs = C * RS;

  auto gload = [&](int c0) {
    const float* inb = In + (size_t)c0 * H * W;
#pragma unroll
    for (int i = 0; i < MAXNI; ++i)
      if (in_lc[i] >= 0)
        in_st[i] = (in_goff[i] >= 0 && c0 + (in_lc[i] >> 20) < C) ? inb[in_goff[i]] : 0.f;
    const float* kbp = Ker + (size_t)c0 * RS;
    const int mlim = (C - c0) * RS;
#pragma unroll
    for (int i = 0; i < MAXNK; ++i) {
      if (ker_km[i] >= 0) {
        const int kl = ker_km[i] >> 16, m = ker_km[i] & 0xffff;
        kvec_t v = (kvec_t)(0.f);
        if (t.k0 + kl < K && m < mlim)
          v = *reinterpret_cast<const kvec_t*>(kbp + (size_t)(t.k0 + kl) * kcs + m);
        ker_st[i] = v;
      }
    }
  };
  auto lstore = [&](int buf) {
    float* lin = lds + buf * g.lds_in_elems;
    float* lk = lds + 2 * g.lds_in_elems + buf * g.lds_ker_elems;
#pragma unroll
    for (int i = 0; i < MAXNI; ++i)
      if (in_lc[i] >= 0) lin[in_lc[i] & 0xfffff] = in_st[i];
#pragma unroll
    for (int i = 0; i < MAXNK; ++i)
      if (ker_km[i] >= 0)
        *reinterpret_cast<kvec_t*>(lk + (ker_km[i] >> 16) * g.ker_rstride + (ker_km[i] & 0xffff)) =
            ker_st[i];
  };
  auto compute = [&](int buf) {
    const float* lin = lds + buf * g.lds_in_elems;
    const float* lk = lds + 2 * g.lds_in_elems + buf * g.lds_ker_elems;
#pragma unroll
    for (int cs = 0; cs < TC / 4; ++cs) {
      // reduction slot gq of the MFMA <-> channel 4*cs + gq at tap (r, s)
      const float* lin_c = lin + (cs * 4 + gq) * g.in_cstride;
      const float* lk_c = lk + (cs * 4 + gq) * RS;
#pragma unroll
      for (int r = 0; r < R; ++r) {
#pragma unroll
        for (int s = 0; s < S; ++s) {
          const int tap = r * g.in_wp + s;
          const int rs = r * S + s;
          float a[WK], b[WP];
#pragma unroll
          for (int kb = 0; kb < WK; ++kb) a[kb] = lk_c[koff[kb] + rs];
#pragma unroll
          for (int pb = 0; pb < WP; ++pb) b[pb] = lin_c[poff[pb] + tap];
#pragma unroll
          for (int kb = 0; kb < WK; ++kb)
#pragma unroll
            for (int pb = 0; pb < WP; ++pb)
              acc[kb][pb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[kb], b[pb], acc[kb][pb], 0, 0, 0);
        }
      }
    }
  };

  gload(0);
  lstore(0);
  __syncthreads();
  for (int ch = 0; ch < g.nchunks; ++ch) {
    const int buf = ch & 1;
    if (ch + 1 < g.nchunks) gload((ch + 1) * TC);
    compute(buf);
    if (ch + 1 < g.nchunks) lstore(buf ^ 1);
    __syncthreads();
  }

  // Epilogue: lane (j, gq) holds Out[k0 + block*16 + 4*gq + v][pixel j].
  const size_t PQ = (size_t)g.P * g.Q;
#pragma unroll
  for (int pb = 0; pb < WP; ++pb) {
    const int px = (wp * WP + pb) * 16 + j;
    const int row_i = px / g.tw, col = px - row_i * g.tw;
    const int rho = t.rho0 + row_i;
    if (px < tpx && rho < t.rho_end && col < t.tw_eff) {
      const int n = rho / g.P, p = rho - n * g.P;
      float* ob = Out + ((size_t)n * K * g.P + p) * g.Q + t.q0 + col;
#pragma unroll
      for (int kb = 0; kb < WK; ++kb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int k = t.k0 + (wk * WK + kb) * 16 + 4 * gq + v;
          if (k < K) ob[(size_t)k * PQ] = acc[kb][pb][v];
        }
    }
  }
}

// ---------------------------------------------------------------------------
// Direct-to-LDS pipeline (gfx950 buffer loads with an LDS destination).
//
// Each buffer load writes its 64 lanes' data to LDS at M0 + lane * width, so
// a wave instruction fills one contiguous 256 B (dword) or 1 KB (dwordx4)
// block of the stage buffer; lanes whose element lies outside the tensor, the
// tile or the channel range pass an offset past the buffer's range and the
// hardware writes zeros.  No VGPRs are used for staging, so NS stages can be
// in flight.  The loads are issued from inline assembly: the compiler then
// does not treat them as LDS writes and does not force a full vmcnt wait
// before every LDS read; instead each step waits for exactly the loads of
// the step it is about to read (loads retire in order) and then barriers.
typedef int v4i __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) float lds_float;

constexpr unsigned kOob = 0x80000000u;  // past every buffer's range (tensors < 2 GB)
constexpr int kStoreNT = 2;  // cache-policy operand of buffer stores: the gfx950 `nt` (streaming) bit

__device__ __forceinline__ v4i make_rsrc(const void* base, unsigned bytes) {
  const unsigned long long p = reinterpret_cast<unsigned long long>(base);
  v4i r;
  r[0] = (int)(unsigned)p;
  r[1] = (int)((unsigned)(p >> 32) & 0xffffu);  // stride 0: raw buffer
  r[2] = (int)bytes;                            // range in bytes
  r[3] = 0x00020000;                            // 32-bit data format
  return r;
}

template <int KV>
__device__ __forceinline__ void dma_load(v4i rsrc, unsigned m0, unsigned voff) {
  if constexpr (KV == 1) {
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds"
                 :: "s"(m0), "v"(voff), "s"(rsrc) : "memory", "m0");
  } else {
    static_assert(KV == 4, "dword or dwordx4");
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :: "s"(m0), "v"(voff), "s"(rsrc) : "memory", "m0");
  }
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // s_waitcnt: vmcnt in bits [3:0] and [15:14]; expcnt and lgkmcnt left at max
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

// The same wait as opaque inline assembly: where compiler-issued loads are
// also in flight, the compiler's wait bookkeeping (which cannot see loads
// issued from inline assembly) might otherwise drop or relax it.
template <int N>
__device__ __forceinline__ void wait_vmcnt_opaque() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Pipeline steps st = (channel group cs, tap rs) of one chunk that the
// phase-skip kernel runs: group cs holds phase f = cs / GPP (GPP groups of
// four channels per phase); with PS false, every step.
template <int NSTEP, int RC, int SC, int GPP, bool PS>
struct PhaseSteps {
  int st[NSTEP > 0 ? NSTEP : 1];
  int n;
  constexpr PhaseSteps() : st{}, n(0) {
    for (int i = 0; i < NSTEP; ++i) {
      const int cs = i / (RC * SC), rs = i % (RC * SC), r = rs / SC, s = rs % SC;
      const int f = PS ? cs / GPP : 0, a = f >> 1, b = f & 1;
      if (PS && ((a == 1 && r == RC - 1) || (b == 1 && s == SC - 1))) continue;
      st[n++] = i;
    }
  }
};

// MF32 selects the inner loop: false, WK x WP blocks of 16x16 on
// v_mfma_f32_16x16x4f32 (four channels per step); true, a 64-row k tile
// (WK = 4) times WP/2 blocks of 32 pixels on v_mfma_f32_32x32x2f32 (two
// channels per step), whose accumulators need no dependency padding and
// which reads half the operand registers per flop.
//
// NWC > 1 splits the reduction inside the workgroup: NWC groups of
// nwk x nwp waves share every staged chunk, group wc taking the channel
// slice [wc * TC / NWC, (wc + 1) * TC / NWC) of each step, and the groups'
// accumulators are summed through LDS at the end (in group order, so the
// result is deterministic).  Small layers then keep every SIMD busy without
// a second, reducing kernel.
//
// PS (phase skip) is for the polyphase rewrite of a stride-2 layer with odd
// taps R = 2 RC - 1, S = 2 SC - 1, run through conv_fwd_ex with In read by
// the phase mapping (four phases (a, b) per input channel).  Tap (r', s') of
// phase (a, b) is a real tap unless a = 1 and r' = RC - 1, or b = 1 and
// s' = SC - 1; the rearranged Ker is zero there (3x3: 7 of 16 taps).  A
// chunk of TC inner channels is laid out phase-major in LDS (position
// f * TC/4 + c holds phase f of the chunk's input channel c), so that each
// step's four channels share one phase, and the steps of zero taps are left
// out of the unrolled loop.
template <int WK, int WP, int NW, int TC, int RC, int SC, int NS, int NLI, int KVI, int NLK, int KVK,
          bool MF32 = false, int NWC = 1, bool PS = false>
__global__ void __launch_bounds__(NW * 64)
conv_f32_dma_kernel(const float* __restrict__ In, const float* __restrict__ Ker,
                    float* __restrict__ Out, const Geom g) {
  static_assert(NS >= 2 && NS <= 4, "pipeline depth");
  static_assert(NWC == 1 || (!MF32 && NW % NWC == 0 && TC % (4 * NWC) == 0),
                "channel groups: 16x16x4 loop, whole waves and whole channel quads per group");
  static_assert(!PS || (!MF32 && NWC == 1 && TC % 16 == 0 && RC > 1 && SC > 1 && KVI == 1 &&
                        (RC * SC) % KVK == 0),
                "phase skip: 16x16x4 loop, four input channels per phase and step, Ker vectors within a tap row");
  constexpr int TCO = TC / 4;  // PS: input channels per chunk
  extern __shared__ __align__(16) float lds[];
  constexpr int IN_REGION = NLI * NW * 64 * KVI;
  constexpr int KER_REGION = NLK * NW * 64 * KVK;
  constexpr int STAGE = IN_REGION + KER_REGION;
  constexpr int L = NLI + NLK;  // loads per wave per step
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int j = lane & 15, gq = lane >> 4;
  constexpr int NWG = NW / NWC;  // waves per channel group
  const int wg = wave % NWG, wc = wave / NWG;
  const int wk = wg % g.nwk, wp = wg / g.nwk;
  const int BK = 16 * WK * g.nwk;
  const int R = RC ? RC : g.R, S = SC ? SC : g.S;
  const int RS = R * S;
  const int H = g.H, W = g.W, C = g.C, K = g.K;
  // Workgroups of channel range r follow those of range r - 1.
  const int split_r = (int)blockIdx.x / g.num_tiles;
  const TileCoord t = tile_coord(g, BK, (int)blockIdx.x - split_r * g.num_tiles);
  const v4i in_rsrc = make_rsrc(In, g.in_bytes);
  const v4i ker_rsrc = make_rsrc(Ker, g.ker_bytes);
  const unsigned lds_base = (unsigned)(size_t)(lds_float*)lds;

  // In loads: instruction i of this wave fills LDS elements
  // [(i*NW + wave)*64*KVI, +64*KVI) of the [TC][in_cstride] In image.
  int in_goff[NLI], in_cl[NLI];
  {
    const int ncols = t.tw_eff + S - 1;
#pragma unroll
    for (int i = 0; i < NLI; ++i) {
      const int e = ((i * NW + wave) * 64 + lane) * KVI;
      in_goff[i] = -1;
      in_cl[i] = 0;
      if (e < TC * g.in_cstride) {
        const int cl = fdiv(e, g.dv_in_cstride), pos = e - cl * g.in_cstride;
        const int row = fdiv(pos, g.dv_in_wp), x = pos - row * g.in_wp;
        if (row < t.nrows && x < ncols) {
          const int nu = t.nu0 + row;
          const int n = fdiv(nu, g.dv_H), y = nu - n * H;
          if (g.nph == 0) {
            in_goff[i] = ((n * C + cl) * H + y) * W + t.q0 + x;
          } else {
            // phase (a, b) of input channel c: a chunk holds whole channels
            // (PS: LDS position cl is phase cl / TCO of channel cl % TCO)
            const int c = PS ? cl % TCO : fdiv(cl, g.dv_nph);
            const int f = PS ? cl / TCO : cl - c * g.nph;
            const int a = fdiv(f, g.dv_nb), b = f - a * g.nb;
            int yi = y, xi = t.q0 + x;
            if (g.Wi) {  // 1x1 kernel view: one row of H' x W' pixels
              yi = fdiv(xi, g.dv_Wi);
              xi -= yi * g.Wi;
            }
            const int iy = yi * g.sh + a - g.ph, ix = xi * g.sw + b - g.pw;
            if (iy >= 0 && iy < g.H0 && ix >= 0 && ix < g.W0) in_goff[i] = ((n * g.C0 + c) * g.H0 + iy) * g.W0 + ix;
            if (PS) in_cl[i] = c * 4 + f;  // the inner channel, for the channel-count check
          }
          if (!PS || g.nph == 0) in_cl[i] = cl;
        }
      }
    }
  }
  // Ker loads: instruction i fills [(i*NW + wave)*64*KVK, +64*KVK) of the
  // [BK][ker_rstride] Ker image.
  const int TCRS = TC * RS;
  int ker_goff[NLK], ker_m[NLK];
#pragma unroll
  for (int i = 0; i < NLK; ++i) {
    const int e = ((i * NW + wave) * 64 + lane) * KVK;
    const int kl = fdiv(e, g.dv_ker_rstride), m = e - kl * g.ker_rstride;
    ker_goff[i] = -1;
    ker_m[i] = 0;
    if (kl < BK && m < TCRS && t.k0 + kl < K) {
      // PS: LDS position (f * TCO + c) * RS + rs holds the rearranged Ker's
      // inner channel c * 4 + f (a vector stays within one channel's taps)
      const int mg = PS ? ((m / RS % TCO) * 4 + m / RS / TCO) * RS + m % RS : m;
      ker_goff[i] = (t.k0 + kl) * C * RS + mg;
      ker_m[i] = mg;
    }
  }
  static_assert(!MF32 || (WK == 4 && WP % 2 == 0), "32x32 blocks: 64 k rows, pixel blocks in pairs of 16");
  constexpr int NPB = MF32 ? WP / 2 : WP;  // pixel blocks of this wave (32 or 16 wide)
  constexpr int BW = MF32 ? 32 : 16;       // block width
  const int l32 = lane & 31, h32 = lane >> 5;
  const int jl = MF32 ? l32 : j;           // this lane's column within a pixel block
  // Per-lane LDS offsets of this lane's output pixel in each pixel block.
  const int tpx = g.tr * g.tw;
  int poff[NPB];
#pragma unroll
  for (int pb = 0; pb < NPB; ++pb) {
    const int px = wp * WP * 16 + pb * BW + jl;
    const int row_i = fdiv(px, g.dv_tw), col = px - row_i * g.tw;
    const int rho = t.rho0 + row_i;
    int off = 0;
    if (px < tpx && rho < t.rho_end && col < t.tw_eff) {
      const int n = fdiv(rho, g.dv_P), p = rho - n * g.P;
      off = (n * H + p - t.nu0) * g.in_wp + col;
    }
    poff[pb] = off;
  }
  constexpr int NKB = MF32 ? 2 : WK;  // k blocks of this wave (32 or 16 rows)
  int koff[NKB];
#pragma unroll
  for (int kb = 0; kb < NKB; ++kb)
    koff[kb] = (MF32 ? wk * 64 + kb * 32 + l32 : (wk * WK + kb) * 16 + j) * g.ker_rstride;

  auto issue = [&](int ch, int slot) {  // pipeline step ch into stage buffer slot % NS
    const int c0 = ch * TC;
    const unsigned stage = lds_base + (unsigned)((slot % NS) * STAGE) * 4u;
    const int coff = g.nph ? fdiv(c0, g.dv_nph) * g.H0 * g.W0 : c0 * H * W;
#pragma unroll
    for (int i = 0; i < NLI; ++i) {
      const unsigned voff =
          (in_goff[i] >= 0 && c0 + in_cl[i] < C) ? (unsigned)(coff + in_goff[i]) * 4u : kOob;
      dma_load<KVI>(in_rsrc, __builtin_amdgcn_readfirstlane(stage + (unsigned)((i * NW + wave) * 64 * KVI) * 4u),
                    voff);
    }
    const int mlim = (C - c0) * RS, kc = c0 * RS;
#pragma unroll
    for (int i = 0; i < NLK; ++i) {
      const unsigned voff =
          (ker_goff[i] >= 0 && ker_m[i] < mlim) ? (unsigned)(kc + ker_goff[i]) * 4u : kOob;
      dma_load<KVK>(ker_rsrc,
                    __builtin_amdgcn_readfirstlane(stage + (unsigned)(IN_REGION + (i * NW + wave) * 64 * KVK) * 4u),
                    voff);
    }
  };

  typedef typename std::conditional<MF32, v16f, v4f>::type acc_t;
  acc_t acc[NKB][NPB];
#pragma unroll
  for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) acc[kb][pb] = acc_t{};

  // One chunk: steps st = (channel group cs, tap r, tap s), a group being four
  // channels (16x16x4) or two (32x32x2).  The operands of step st+1 are read
  // from LDS before the MFMAs of step st are issued, so LDS latency overlaps
  // the matrix core instead of stalling it.
  static_assert(RC > 0 && SC > 0, "compile-time taps");
  constexpr int CG = MF32 ? 2 : 4;  // channels per step
  constexpr int NSTEP = (TC / CG / NWC) * RC * SC;
  const int cl = MF32 ? h32 : gq;   // this lane's channel within a group
  auto compute = [&](int buf) {
    // this wave's channel slice of the chunk
    const float* lin = lds + buf * STAGE + wc * (TC / NWC) * g.in_cstride;
    const float* lk = lds + buf * STAGE + IN_REGION + wc * (TC / NWC) * RS;
    float a[2][NKB], b[2][NPB];
    auto fetch = [&](int st, int slot) {
      const int cs = st / (RC * SC), rs = st % (RC * SC);
      const int r = rs / SC, s = rs % SC;
      const float* lin_c = lin + (cs * CG + cl) * g.in_cstride + r * g.in_wp + s;
      const float* lk_c = lk + (cs * CG + cl) * RS + rs;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) a[slot][kb] = lk_c[koff[kb]];
#pragma unroll
      for (int pb = 0; pb < NPB; ++pb) b[slot][pb] = lin_c[poff[pb]];
    };
    // PS: only the steps of real taps, in order (see the template's comment)
    constexpr PhaseSteps<NSTEP, RC, SC, TCO / 4, PS> steps{};
    fetch(steps.st[0], 0);
#pragma unroll
    for (int i = 0; i < steps.n; ++i) {
      const int cur = i & 1;
      if (i + 1 < steps.n) fetch(steps.st[i + 1], cur ^ 1);
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb) {
          if constexpr (MF32)
            acc[kb][pb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[cur][kb], b[cur][pb], acc[kb][pb], 0, 0, 0);
          else
            acc[kb][pb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[cur][kb], b[cur][pb], acc[kb][pb], 0, 0, 0);
        }
    }
  };

  // This workgroup's channel range: pipeline steps [ch0, ch0 + nch).  All
  // NS stage buffers are filled up front (a short reduction is then one
  // round trip to memory, not one per step); from the second step on, each
  // iteration refills the buffer the previous one computed, which the
  // barrier has freed, so NS - 1 steps stay in flight behind the current one.
  const int ch0 = split_r * g.cps;
  const int nch = min(g.cps, g.nchunks - ch0);
#pragma unroll
  for (int s = 0; s < NS; ++s)
    if (s < nch) issue(ch0 + s, s);
  for (int ch = 0; ch < nch; ++ch) {
    // wait for this step's loads: the later steps already issued may stay in
    // flight (loads retire in order)
    const int ahead = min(ch == 0 ? NS - 1 : NS - 2, nch - 1 - ch);
    if (ahead >= 3) wait_vmcnt<(3 * L < 64 ? 3 * L : 63)>();
    else if (ahead == 2) wait_vmcnt<(2 * L < 64 ? 2 * L : 63)>();
    else if (ahead == 1) wait_vmcnt<(L < 64 ? L : 63)>();
    else wait_vmcnt<0>();
    __syncthreads();
    if (ch >= 1 && ch + NS - 1 < nch) issue(ch0 + ch + NS - 1, ch + NS - 1);
    compute(ch % NS);
  }

  // Epilogue: lane (j, gq) holds Out[k0 + block*16 + 4*gq + v][pixel j]
  // (16x16x4), lane (l32, h32) rows 8*(v/4) + 4*h32 + v%4 of pixel l32
  // (32x32x2); a split plan writes range split_r's partial sums to slice
  // split_r of the workspace passed as Out.
  const size_t PQ = (size_t)g.P * g.Q;
  if constexpr (NWC > 1) {
    // Every wave parks its accumulators in LDS, register r of wave w at
    // [(w * NREG + r) * 64 + lane]; then the wave of group wc sums registers
    // [wc * NREG / NWC, (wc + 1) * NREG / NWC) over the groups in order and
    // stores them.  The last step's loads have all landed (vmcnt 0 above),
    // and the barrier keeps the pipeline's last reads before the writes.
    constexpr int NREG = NKB * NPB * 4;
    constexpr int RPW = NREG / NWC;
    static_assert(NREG % NWC == 0, "registers per group");
    static_assert(NW * NREG * 64 <= NS * STAGE, "reduction fits the pipeline's LDS");
    __syncthreads();
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
        for (int v = 0; v < 4; ++v) lds[(wave * NREG + (kb * NPB + pb) * 4 + v) * 64 + lane] = acc[kb][pb][v];
    __syncthreads();
    for (int i = 0; i < RPW; ++i) {
      const int r = wc * RPW + i;
      const int kb = r / (NPB * 4), pb = (r / 4) % NPB, v = r % 4;
      float sum = lds[(wg * NREG + r) * 64 + lane];
#pragma unroll
      for (int c = 1; c < NWC; ++c) sum += lds[((c * NWG + wg) * NREG + r) * 64 + lane];
      const int px = wp * WP * 16 + pb * 16 + j;
      const int row_i = fdiv(px, g.dv_tw), col = px - row_i * g.tw;
      const int rho = t.rho0 + row_i;
      const int k = t.k0 + (wk * WK + kb) * 16 + 4 * gq + v;
      if (px < tpx && rho < t.rho_end && col < t.tw_eff && k < K) {
        const int n = fdiv(rho, g.dv_P), p = rho - n * g.P;
        Out[(size_t)split_r * g.N * K * PQ + (((size_t)n * K + k) * g.P + p) * g.Q + t.q0 + col] = sum;
      }
    }
    return;
  }
#pragma unroll
  for (int pb = 0; pb < NPB; ++pb) {
    const int px = wp * WP * 16 + pb * BW + jl;
    const int row_i = fdiv(px, g.dv_tw), col = px - row_i * g.tw;
    const int rho = t.rho0 + row_i;
    if (px < tpx && rho < t.rho_end && col < t.tw_eff) {
      const int n = fdiv(rho, g.dv_P), p = rho - n * g.P;
      float* ob = Out + (size_t)split_r * g.N * K * PQ + ((size_t)n * K * g.P + p) * g.Q + t.q0 + col;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        if constexpr (MF32) {
          // register v holds row 8*(v/4) + 4*h32 + v%4 of the 32-row block
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int k = t.k0 + wk * 64 + kb * 32 + 8 * (v / 4) + 4 * h32 + v % 4;
            if (k < K) ob[(size_t)k * PQ] = acc[kb][pb][v];
          }
        } else {
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int k = t.k0 + (wk * WK + kb) * 16 + 4 * gq + v;
            if (k < K) ob[(size_t)k * PQ] = acc[kb][pb][v];
          }
        }
      }
    }
  }
}

// Compile-time loop: f(std::integral_constant<int, i>) for i = 0..N-1, each
// call inlined with its own constant (a plain unroll pragma gives up on long
// bodies, and a rolled loop would index register arrays dynamically).
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// ---------------------------------------------------------------------------
// bf16 inputs, fp32 accumulation (16x16x32 bf16 MFMA).
//
// The MFMA's 32-deep reduction is one tap (r, s) of 32 input channels, so
// both operands must hold 8 consecutive channels per lane.  In arrives as
// NCHW; the staging step transposes a tile into a channel-fastest LDS image
// [row][pixel][32 channels] (64 B per pixel, four 16 B chunks of 8 channels,
// chunk index XOR-swizzled with pixel bits so that 16 lanes reading 16
// neighbouring pixels touch every bank pair once).  Ker is held in LDS for the
// whole kernel as [k][tap][32 channels] (same chunk swizzle by k).  Each
// workgroup is persistent over every G-th tile (G workgroups); while it
// computes one tile, the global loads of its next tile's In are in flight in
// registers.  Per tile: stage, barrier, MFMAs, stores.
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef unsigned short v8u16 __attribute__((ext_vector_type(8)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int chunk_swz(int chunk, int idx) { return chunk ^ ((idx >> 1) & 3); }

template <int WK, int WP, int RC, int SC, int MAXIT>
__global__ void __launch_bounds__(kThreads)
conv_bf16_kernel(const unsigned short* __restrict__ In, const unsigned short* __restrict__ Ker,
                 float* __restrict__ Out, const Geom g) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int TC = 32;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int j = lane & 15, gq = lane >> 4;
  const int wk = wave % g.nwk, wp = wave / g.nwk;
  const int BK = 16 * WK * g.nwk;
  const int R = RC, S = SC, RS = RC * SC;
  const int H = g.H, W = g.W, C = g.C, K = g.K, P = g.P, Q = g.Q;
  // LDS: Ker [BK][kpitch taps][64 B], then In [in_rows][in_wp pixels][64 B]
  const int kpitch = (RS & 1) ? RS : RS + 1;
  unsigned char* lker = smem;
  unsigned char* lin = smem + (size_t)BK * kpitch * 64;
  const int tiles = g.tiles_rows * g.tiles_cols * g.tiles_k;
  const int G = gridDim.x;
  const int L = xcd_remap(blockIdx.x, G);
  // tiles L, L + G, L + 2G, ...: at any time the workgroups work on
  // neighbouring tiles (see the transposing kernel below)
  const int t_begin = L, t_end = tiles;
  if (t_begin >= t_end) return;
  const int nchunks = (C + TC - 1) / TC;
  const bool resident = (nchunks == 1) && (g.tiles_k == 1);

  auto tile_of = [&](int T, int& kt, int& ct, int& rt) {
    kt = T % g.tiles_k;
    const int rest = T / g.tiles_k;
    ct = rest % g.tiles_cols;
    rt = rest / g.tiles_cols;
  };

  // Ker staging for channel chunk c0 and k tile k0: items (kl, tap, octet).
  auto stage_ker = [&](int k0, int c0) {
    const int items = BK * RS * 4;
    for (int it = tid; it < items; it += kThreads) {
      const int o = it & 3, rest = it >> 2;
      const int rs = rest % RS, kl = rest / RS;
      v8u16 v;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int c = c0 + 8 * o + e, k = k0 + kl;
        v[e] = (c < C && k < K) ? Ker[((size_t)k * C + c) * RS + rs] : (unsigned short)0;
      }
      *reinterpret_cast<v8u16*>(lker + ((size_t)kl * kpitch + rs) * 64 + chunk_swz(o, kl) * 16) = v;
    }
  };

  // In staging through registers: items (octet o, halo row, pixel pair).
  const int in_wp = g.in_wp;             // halo columns, even
  const int npair = in_wp >> 1;
  const int in_items = 4 * g.in_rows * npair;
  unsigned st_lo[MAXIT][8];              // per item: 8 channels x 2 pixels (packed pairs)
  auto gload_in = [&](int T, int c0) {
    int kt, ct, rt;
    tile_of(T, kt, ct, rt);
    const int NP = g.N * P;
    const int rho0 = rt * g.tr, rho_end = min(rho0 + g.tr, NP);
    const int q0 = ct * g.tw, ncols = min(g.tw, Q - q0) + S - 1;
    const int nf = rho0 / P, nu0 = nf * H + (rho0 - nf * P);
    const int nl = (rho_end - 1) / P, nrows = nl * H + (rho_end - 1 - nl * P) + R - nu0;
    const bool even = ((W | q0) & 1) == 0 && (reinterpret_cast<uintptr_t>(In) & 3) == 0;
#pragma unroll
    for (int m = 0; m < MAXIT; ++m) {
      const int it = tid + m * kThreads;
      const int o = it / (g.in_rows * npair), rest = it - o * (g.in_rows * npair);
      const int row = rest / npair, x = (rest - row * npair) * 2;
      const bool ok = it < in_items && row < nrows;
      const int nu = nu0 + row;
      const int n = nu / H, y = nu - n * H;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int c = c0 + 8 * o + e;
        unsigned v = 0;
        if (ok && c < C && x < ncols) {
          const size_t base = (((size_t)n * C + c) * H + y) * W + q0 + x;
          if (even && x + 1 < ncols) {
            v = *reinterpret_cast<const unsigned*>(In + base);
          } else {
            v = In[base];
            if (x + 1 < ncols) v |= (unsigned)In[base + 1] << 16;
          }
        }
        st_lo[m][e] = v;
      }
    }
  };
  auto lstore_in = [&]() {
#pragma unroll
    for (int m = 0; m < MAXIT; ++m) {
      const int it = tid + m * kThreads;
      if (it < in_items) {
        const int o = it / (g.in_rows * npair), rest = it - o * (g.in_rows * npair);
        const int row = rest / npair, x = (rest - row * npair) * 2;
        v4u p0, p1;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const unsigned a = st_lo[m][2 * e], b = st_lo[m][2 * e + 1];
          p0[e] = (a & 0xffffu) | (b << 16);          // pixel x: channels 2e, 2e+1
          p1[e] = (a >> 16) | (b & 0xffff0000u);      // pixel x+1
        }
        const int px0 = row * in_wp + x, px1 = px0 + 1;
        *reinterpret_cast<v4u*>(lin + (size_t)px0 * 64 + chunk_swz(o, px0) * 16) = p0;
        *reinterpret_cast<v4u*>(lin + (size_t)px1 * 64 + chunk_swz(o, px1) * 16) = p1;
      }
    }
  };

  if (resident) {
    stage_ker(0, 0);
  }
  if (resident) gload_in(t_begin, 0);
  for (int T = t_begin; T < t_end; T += G) {
    int kt, ct, rt;
    tile_of(T, kt, ct, rt);
    const int NP = g.N * P;
    const int rho0 = rt * g.tr, rho_end = min(rho0 + g.tr, NP);
    const int q0 = ct * g.tw, tw_eff = min(g.tw, Q - q0);
    const int k0 = kt * BK;
    const int nf = rho0 / P, nu0 = nf * H + (rho0 - nf * P);
    const int tpx = g.tr * g.tw;
    int poff[WP];
#pragma unroll
    for (int pb = 0; pb < WP; ++pb) {
      const int px = (wp * WP + pb) * 16 + j;
      const int row_i = px / g.tw, col = px - row_i * g.tw;
      const int rho = rho0 + row_i;
      int off = 0;
      if (px < tpx && rho < rho_end && col < tw_eff) {
        const int n = rho / P, p = rho - n * P;
        off = (n * H + p - nu0) * in_wp + col;
      }
      poff[pb] = off;
    }
    v4f acc[WK][WP];
#pragma unroll
    for (int kb = 0; kb < WK; ++kb)
#pragma unroll
      for (int pb = 0; pb < WP; ++pb) acc[kb][pb] = v4f{0.f, 0.f, 0.f, 0.f};

    for (int ch = 0; ch < nchunks; ++ch) {
      __syncthreads();  // previous users of the LDS buffers are done
      if (!resident) {
        stage_ker(k0, ch * TC);
        gload_in(T, ch * TC);
      }
      lstore_in();
      __syncthreads();
      if (resident && T + G < t_end) gload_in(T + G, 0);  // in flight during the MFMAs
#pragma unroll
      for (int r = 0; r < R; ++r) {
#pragma unroll
        for (int s = 0; s < S; ++s) {
          v8bf a[WK], b[WP];
#pragma unroll
          for (int kb = 0; kb < WK; ++kb) {
            const int kl = (wk * WK + kb) * 16 + j;
            a[kb] = *reinterpret_cast<const v8bf*>(lker + ((size_t)kl * kpitch + r * S + s) * 64 +
                                                  chunk_swz(gq, kl) * 16);
          }
#pragma unroll
          for (int pb = 0; pb < WP; ++pb) {
            const int pp = poff[pb] + r * in_wp + s;
            b[pb] = *reinterpret_cast<const v8bf*>(lin + (size_t)pp * 64 + chunk_swz(gq, pp) * 16);
          }
#pragma unroll
          for (int kb = 0; kb < WK; ++kb)
#pragma unroll
            for (int pb = 0; pb < WP; ++pb)
              acc[kb][pb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[kb], b[pb], acc[kb][pb], 0, 0, 0);
        }
      }
    }
    // Epilogue: lane (j, gq) holds Out[k0 + block*16 + 4*gq + v][pixel j].
    const size_t PQ = (size_t)P * Q;
#pragma unroll
    for (int pb = 0; pb < WP; ++pb) {
      const int px = (wp * WP + pb) * 16 + j;
      const int row_i = px / g.tw, col = px - row_i * g.tw;
      const int rho = rho0 + row_i;
      if (px < tpx && rho < rho_end && col < tw_eff) {
        const int n = rho / P, p = rho - n * P;
        float* ob = Out + ((size_t)n * K * P + p) * Q + q0 + col;
#pragma unroll
        for (int kb = 0; kb < WK; ++kb)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int k = k0 + (wk * WK + kb) * 16 + 4 * gq + v;
            if (k < K) ob[(size_t)k * PQ] = acc[kb][pb][v];
          }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 kernel for C = 32 (one 16x16x32 MFMA covers the whole channel range),
// K <= 64, taps RC x SC (SC <= 3), W even, tile columns a multiple of 16.
//
// The MFMA operand that carries In wants eight consecutive channels of one
// pixel per lane, while In is NCHW.  Rather than transposing In into a
// channel-fastest tile, the tile stays pixel-fastest in LDS
// ([copy][c][row][x], row-major as in memory) and the transposing LDS read of
// gfx950 (ds_read_b64_tr_b16) produces the operand: within each 16-lane
// group, source lane s reads four consecutive pixels 4*(s%4).. of channel
// 4h + s/4 (plus the group's channel octet), and lane i receives pixel i of
// channels 4h..4h+3.  Those reads must be 8-byte aligned, so each tap column
// s has its own copy of the tile, shifted by s pixels (copy s at x holds pixel
// x + s); every channel plane is padded so the four channels of one read fall
// on distinct banks.
//
// The In operand is the MFMA's A side (rows = pixels) and Ker its B side
// (columns = k), so each lane ends with four consecutive pixels of one k and
// stores them as one 16-byte vector.
//
// The Ker slice (64 k rows) stays in LDS for the whole kernel: it is read
// once with 16-byte loads in its natural [k][c][r][s] order and scattered
// into [k][tap][8 octets of channels, swizzled] while the first tile's In
// loads are in flight.  Workgroups are persistent over every G-th tile.
// Each tile's In rows are loaded into registers while the previous tile
// computes (16-byte loads away from the right image edge), then written as
// the SC shifted copies (copy 1 is the funnel shift of neighbouring dwords).
//
// Every workgroup does the same work per tile, so if a tile's results were
// stored in one burst after its last MFMA, all CUs would store at once and
// leave HBM idle while they compute.  Instead each wave computes its tile in
// NPART parts (groups of pixel blocks); the stores of one part are spread
// over the MFMAs of the next part (the last part's over the first part of the
// next tile), which keeps writes flowing during the whole kernel.
typedef short v4s __attribute__((ext_vector_type(4)));
typedef short v8s __attribute__((ext_vector_type(8)));

template <int TR, int TW, int RC, int SC, bool OUTB>
__global__ void __launch_bounds__(kThreads)
conv_bf16_tr_kernel(const unsigned short* __restrict__ In, const unsigned short* __restrict__ Ker,
                    float* __restrict__ Out, const Geom g) {
  // OUTB: Out holds bf16 (the fp32 sums rounded to nearest even) instead of fp32
  static_assert(SC >= 1 && SC <= 3, "copies from two neighbouring dwords");
  static_assert(TW % 16 == 0 && (TR * (TW / 16)) % 4 == 0, "whole blocks of 16 for four waves");
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int RS = RC * SC;
  constexpr int KPITCH = (RS & 1) ? RS : RS + 1;  // Ker taps per row (odd: conflict-free rows)
  constexpr int KER_BYTES = 64 * KPITCH * 64;
  constexpr int IN_ROWS = TR + RC - 1;            // tiles never straddle images (P % TR == 0)
  constexpr int CP = IN_ROWS * TW + (16 - (IN_ROWS * TW) % 64 + 64) % 64;  // plane: 16 (mod 64) elements
  static_assert(CP % 64 == 16 && CP >= IN_ROWS * TW, "channel plane padding");
  constexpr int GPR = TW / 8;                     // groups of four dwords (8 pixels) per tile row
  constexpr int TPR = 32 * GPR;                   // threads covering one row of all 32 channels
  static_assert(kThreads % TPR == 0, "whole rows per pass");
  constexpr int RPT = kThreads / TPR;             // rows per pass
  constexpr int NIT = (IN_ROWS + RPT - 1) / RPT;  // items per thread
  constexpr int CBR = TW / 16;                    // blocks per tile row
  constexpr int WP = TR * CBR / 4;                // blocks per wave
  constexpr int NPART = WP % 2 == 0 ? 2 : 1;      // parts per tile
  constexpr int PB = WP / NPART;                  // blocks per part
  constexpr int NST = PB * 4;                     // (block, k block) stores per part
  constexpr int KV = 64 * 32 * RS / 8;            // 16-byte vectors of a 64-row Ker slice
  constexpr int NKV = KV / kThreads;
  static_assert(KV % kThreads == 0, "whole Ker vectors per thread");
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int j = lane & 15, gq = lane >> 4;
  const int H = g.H, W = g.W, K = g.K, P = g.P, Q = g.Q;
  unsigned char* lker = smem;
  unsigned short* lin = reinterpret_cast<unsigned short*>(smem + KER_BYTES);
  const int tiles = g.tiles_rows * g.tiles_cols;
  const int G = gridDim.x;
  const int L = xcd_remap(blockIdx.x, G);
  // Workgroup L takes tiles L, L + G, L + 2G, ...  At any time the grid
  // works on G consecutive tiles, which cover whole rows of every Out plane:
  // HBM receives the writes (and serves the In rows, halos shared through
  // the L2) of one compact region instead of G scattered ones.  Measured on
  // the 226^2 layer with In from HBM, 14-20% faster than contiguous ranges.
  const int t_begin = L, t_end = tiles;
  if (t_begin >= t_end) return;
  // vector output stores (4 pixels: 16 bytes, or 8 for bf16 Out) need
  // Q % 4 == 0 and an Out aligned to that size
  constexpr int OUT_E = OUTB ? 2 : 4;
  const bool vec_out = (Q & 3) == 0 && (reinterpret_cast<uintptr_t>(Out) & (4 * OUT_E - 1)) == 0;
  // bf16 Out in 16-byte pieces of two neighbouring blocks (see the stores)
  constexpr bool PAIRED = OUTB && PB % 2 == 0 && CBR % 2 == 0;
  const bool pair_out = PAIRED && (Q & 7) == 0 && (reinterpret_cast<uintptr_t>(Out) & 15) == 0;

  // Ker loads first (rows past K read zeros: past the buffer's range)
  const __amdgpu_buffer_rsrc_t krsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<unsigned short*>(Ker), (short)0, (int)g.ker_bytes, 0x00020000);
  v4u kv[NKV];
#pragma unroll
  for (int i = 0; i < NKV; ++i) {
    const int v = tid + i * kThreads;
    kv[i] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(krsrc, 16u * v, 0, 0));
  }
  __builtin_amdgcn_sched_barrier(0);  // all Ker loads ahead of the first tile's

  // Tile T: output rows [p0, p0 + TR) of image n, columns [q0, q0 + TW).
  auto tile_start = [&](int T, int& n, int& p0, int& q0) __attribute__((always_inline)) {
    const int ct = T % g.tiles_cols, rt = T / g.tiles_cols;
    const int rho0 = rt * TR;
    n = rho0 / P;
    p0 = rho0 - n * P;
    q0 = ct * TW;
  };

  // In rows of a tile -> registers.  Thread tid loads channel ic, group gr
  // of four dwords (pixels x = q0+8gr .. x+9: dwords 4gr .. 4gr+4, the last
  // one for the shifted copies) of rows irow0, irow0 + RPT, ...: per row one
  // 16-byte load of pixels x .. x+7 and one 4-byte load of x+8, x+9.  A
  // thread whose group crosses the right edge of the row (x < W < x + 8)
  // loads the last 8 pixels of the row instead and keeps the number of dwords
  // it moved back (sh = (x + 8 - W) / 2); the LDS write moves them forward
  // again, with zeros past the row.  Groups wholly past the row read zeros.
  // (W >= 8 keeps that load inside the row.)
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<unsigned short*>(In), (short)0, (int)g.in_bytes, 0x00020000);
  const int gr = tid % GPR, ic = (tid / GPR) % 32, irow0 = tid / TPR;
  v4u q[NIT];
  unsigned d4[NIT];
  unsigned sh = 0;
  auto gload = [&](int T) __attribute__((always_inline)) {
    // a tile past the end loads nothing (every offset past the range), so
    // the loop issues the same memory instructions on every pass
    const bool tv = T < t_end;
    int n, p0, q0;
    tile_start(tv ? T : t_begin, n, p0, q0);
    const int x = q0 + 8 * gr;
    const int over = max(0, x + 8 - W);  // pixels past the row end (even; < 8 when x < W)
    sh = (unsigned)over >> 1;
    // element offset of (n, ic, p0 + irow0, x)
    const unsigned base = (unsigned)(((n * 32 + ic) * H + p0 + irow0) * W + x) * 2u;
#pragma unroll
    for (int i = 0; i < NIT; ++i) {
      const bool ok = tv && irow0 + RPT * i < IN_ROWS && x < W;
      const unsigned off = base + (unsigned)(RPT * i * W) * 2u;
      q[i] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rsrc, ok ? off - 2u * over : kOob, 0, 0));
      d4[i] = __builtin_amdgcn_raw_buffer_load_b32(rsrc, ok && x + 8 < W ? off + 16u : kOob, 0, 0);
    }
  };
  auto lstore = [&](auto&& after_item) __attribute__((always_inline)) {
    static_for<NIT>([&](auto ic_) __attribute__((always_inline)) {
      constexpr int i = decltype(ic_)::value;
      const int row = irow0 + RPT * i;
      if (row < IN_ROWS) {
        unsigned dw[5];
        dw[0] = sh == 0 ? q[i][0] : sh == 1 ? q[i][1] : sh == 2 ? q[i][2] : q[i][3];
        dw[1] = sh == 0 ? q[i][1] : sh == 1 ? q[i][2] : sh == 2 ? q[i][3] : 0u;
        dw[2] = sh == 0 ? q[i][2] : sh == 1 ? q[i][3] : 0u;
        dw[3] = sh == 0 ? q[i][3] : 0u;
        dw[4] = d4[i];
        v4u* dst = reinterpret_cast<v4u*>(lin + ic * CP + row * TW + 8 * gr);  // 16-byte aligned
        dst[0] = v4u{dw[0], dw[1], dw[2], dw[3]};  // copy 0: pixel x
        if constexpr (SC > 1) {                    // copy 1: x + 1
          v4u v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = (dw[e] >> 16) | (dw[e + 1] << 16);
          dst[32 * CP / 8] = v;
        }
        if constexpr (SC > 2) dst[32 * CP / 4] = v4u{dw[1], dw[2], dw[3], dw[4]};  // copy 2: x + 2
      }
      after_item(ic_);
    });
  };

  gload(t_begin);
  __builtin_amdgcn_sched_barrier(0);  // both sets of loads in flight before the Ker staging waits
  // Ker -> LDS [k][tap][octet of channels, swizzled][8], through the (still
  // unused) In region: the natural order first, with 16-byte writes, then
  // each thread gathers the eight channels of one (k, tap, octet) and writes
  // them as one 16-byte chunk (scattering single elements straight from the
  // loaded vectors hit the same banks from many lanes).
  static_assert(64 * 32 * RS * 2 <= SC * 32 * CP * 2, "Ker staging fits the In region");
#pragma unroll
  for (int i = 0; i < NKV; ++i) reinterpret_cast<v4u*>(lin)[tid + i * kThreads] = kv[i];
  __syncthreads();
  for (int it = tid; it < 64 * RS * 4; it += kThreads) {
    const int o = it & 3, rest = it >> 2;
    const int rs = rest % RS, kl = rest / RS;
    const unsigned short* src = lin + (kl * 32 + 8 * o) * RS + rs;  // element (kl, 8o + e, rs) at e*RS
    v8u16 val;
#pragma unroll
    for (int e = 0; e < 8; ++e) val[e] = src[e * RS];
    *reinterpret_cast<v8u16*>(lker + ((size_t)kl * KPITCH + rs) * 64 + chunk_swz(o, kl) * 16) = val;
  }

  // Results of the previous part, stored while the current part computes.
  // Lane (j, gq) holds Out[k = 16*kb + j][pixels 4*gq .. 4*gq+3 of block bi].
  // Buffer stores with 32-bit offsets (Out < 2 GB); a masked lane's offset is
  // past the buffer's range, where the store is dropped.  The stores go k
  // block by k block, so the blocks of one tile row (neighbouring pieces of
  // the same Out lines) leave one after another; plain stores, no streaming
  // hint (with In from HBM the hint cost 2-10% on the 226^2 layer).
  const __amdgpu_buffer_rsrc_t orsrc = __builtin_amdgcn_make_buffer_rsrc(
      Out, (short)0, (int)((unsigned)g.N * K * P * Q * (unsigned)OUT_E), 0x00020000);
  v4f pend[PB][4];
  bool have_pend = false;
  int pbase = 0, pcol = 0, ppart = 0;  // element offset of (n, k = j, row p0, column q0 + 4 gq)
  auto store_pend = [&](auto si, auto fast) __attribute__((always_inline)) {
    constexpr int bi = decltype(si)::value % PB, kb = decltype(si)::value / PB;
    const int b = wave * WP + ppart * PB + bi;
    const int col = pcol + 16 * (b % CBR);
    const bool ok = have_pend && kb * 16 + j < K;
    const unsigned el = (unsigned)(pbase + kb * 16 * P * Q + (b / CBR) * Q + 16 * (b % CBR));
    if constexpr (OUTB) {
      // Round to bf16 (nearest even; the conversion instruction of gfx950).
      // Four pixels of bf16 are only 8 bytes, and 32-byte pieces of a line
      // write slowly; so two neighbouring blocks are stored together: lane
      // pairs (gq, gq ^ 1) swap halves through ds_bpermute, and each lane
      // stores 8 consecutive pixels (16 bytes): even gq those of block bi,
      // odd gq those of block bi + 1, 64 bytes per k row.  Needs Q % 8 == 0
      // and a 16-byte aligned Out; otherwise 2-byte stores per pixel.
      auto cvt = [](const v4f& a, unsigned& lo, unsigned& hi) __attribute__((always_inline)) {
        unsigned short h[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) h[v] = __builtin_bit_cast(unsigned short, (__bf16)a[v]);
        lo = (unsigned)h[0] | ((unsigned)h[1] << 16);
        hi = (unsigned)h[2] | ((unsigned)h[3] << 16);
      };
      if constexpr (decltype(fast)::value) {
        if constexpr (PAIRED && bi % 2 == 0) {
          unsigned a0, a1, b0, b1;
          cvt(pend[bi][kb], a0, a1);
          cvt(pend[bi + 1][kb], b0, b1);
          const bool even = (gq & 1) == 0;
          const int partner = (lane ^ 16) * 4;
          const unsigned r0 = (unsigned)__builtin_amdgcn_ds_bpermute(partner, (int)(even ? b0 : a0));
          const unsigned r1 = (unsigned)__builtin_amdgcn_ds_bpermute(partner, (int)(even ? b1 : a1));
          const v4u w = even ? v4u{a0, a1, r0, r1} : v4u{r0, r1, b0, b1};
          const unsigned e8 = even ? el : el + 12u;  // odd: block bi + 1, pixels 4 (gq - 1) ..
          const int c8 = even ? col : col + 12;
          __builtin_amdgcn_raw_buffer_store_b128(w, orsrc, ok && c8 < Q ? e8 * 2u : kOob, 0, 0);
        }
      } else {
        const v4f a = pend[bi][kb];
#pragma unroll
        for (int v = 0; v < 4; ++v)
          __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, (__bf16)a[v]), orsrc,
                                                ok && col + v < Q ? (el + v) * 2u : kOob, 0, 0);
      }
    } else {
      const unsigned off = el * 4u;
      if constexpr (decltype(fast)::value) {
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, pend[bi][kb]), orsrc,
                                               ok && col < Q ? off : kOob, 0, 0);
      } else {
        // (the whole vector is reinterpreted: a bit cast of one element
        // lvalue of a vector compiles to element 0 for every v)
        const v4u pv = __builtin_bit_cast(v4u, pend[bi][kb]);
#pragma unroll
        for (int v = 0; v < 4; ++v)
          __builtin_amdgcn_raw_buffer_store_b32(pv[v], orsrc, ok && col + v < Q ? off + 4u * v : kOob, 0, 0);
      }
    }
  };

  // transposing-read source of this lane: channel 8*gq + 4h + s/4, pixels
  // 4*(s%4).. of the block (s = lane % 16)
  const int src_c = 8 * gq + j / 4, src_x = 4 * (j % 4);
  // The last part's stores: the first NST_COPY during the LDS copy phase
  // (one or two per item), the rest over the first part's taps; HBM then
  // receives writes during the copies too.
  constexpr int NST_COPY = NST / 2;
  // The tile loop is instantiated once per store path (vector stores, or
  // the narrow fallback for an unaligned Out or Q % 4 != 0) and the path is
  // chosen once.  The loop is rotated (each pass: the MFMAs of tile T, then
  // the copies of tile T + G, then the loads of tile T + 2G), and it issues
  // the same memory instructions on every pass: so the path from a tile's
  // loads to their use is the same on entry and around the loop, and the
  // compiler's waits for the In loads count the stores issued after them
  // instead of waiting for every store to complete.
  auto run = [&](auto fast) __attribute__((always_inline)) {
    // the next tile's In copies (zeros past the last tile), with the first
    // NST_COPY stores of the previous part
    auto copy_phase = [&]() __attribute__((always_inline)) {
      __syncthreads();  // every wave is done reading the copies (and the Ker writes)
      lstore([&](auto ic_) __attribute__((always_inline)) {
        constexpr int i = decltype(ic_)::value;
        constexpr int s0 = i * NST_COPY / NIT, s1 = (i + 1) * NST_COPY / NIT;
        static_for<s1 - s0>([&](auto si) __attribute__((always_inline)) {
          store_pend(std::integral_constant<int, s0 + decltype(si)::value>{}, fast);
        });
      });
      __syncthreads();
    };
    copy_phase();
    gload(t_begin + G);
    for (int T = t_begin; T < t_end; T += G) {
      int n, p0, q0;
      tile_start(T, n, p0, q0);
      static_for<NPART>([&](auto part) __attribute__((always_inline)) {
        v4f acc[PB][4];
#pragma unroll
        for (int bi = 0; bi < PB; ++bi)
#pragma unroll
          for (int kb = 0; kb < 4; ++kb) acc[bi][kb] = v4f{0.f, 0.f, 0.f, 0.f};
        static_for<RS>([&](auto rsc) __attribute__((always_inline)) {
          constexpr int rs = decltype(rsc)::value, r = rs / SC, sx = rs % SC;
          v8bf kop[4];
#pragma unroll
          for (int kb = 0; kb < 4; ++kb) {
            const int kl = kb * 16 + j;
            kop[kb] = *reinterpret_cast<const v8bf*>(lker + ((size_t)kl * KPITCH + rs) * 64 + chunk_swz(gq, kl) * 16);
          }
          // block bi's In operand: block b = tile row b / CBR, columns 16 * (b % CBR) ..
          auto read_iop = [&](int bi) __attribute__((always_inline)) {
            const int b = wave * WP + decltype(part)::value * PB + bi;
            const unsigned short* src =
                lin + sx * 32 * CP + src_c * CP + (b / CBR + r) * TW + 16 * (b % CBR) + src_x;
            const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)(src));
            const v4s hi =
                __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)(src + 4 * CP));
            return __builtin_bit_cast(v8bf, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
          };
          if constexpr (NPART == 1) {
            // one part per tile (an odd number of blocks per wave): every
            // block's operand is read first, then the MFMAs (measured 3-7%
            // faster on the 14x32 and 7x64 tilings; slower with two parts)
            v8bf iop[PB];
#pragma unroll
            for (int bi = 0; bi < PB; ++bi) iop[bi] = read_iop(bi);
#pragma unroll
            for (int bi = 0; bi < PB; ++bi)
#pragma unroll
              for (int kb = 0; kb < 4; ++kb)
                acc[bi][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(iop[bi], kop[kb], acc[bi][kb], 0, 0, 0);
          } else {
#pragma unroll
            for (int bi = 0; bi < PB; ++bi) {
              const v8bf iop = read_iop(bi);
#pragma unroll
              for (int kb = 0; kb < 4; ++kb)
                acc[bi][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(iop, kop[kb], acc[bi][kb], 0, 0, 0);
            }
          }
          // this tap's share of the previous part's stores (for the first
          // part, those not issued during the copies)
          constexpr int SB = decltype(part)::value == 0 ? NST_COPY : 0;
          constexpr int s0 = SB + rs * (NST - SB) / RS, s1 = SB + (rs + 1) * (NST - SB) / RS;
          static_for<s1 - s0>([&](auto si) __attribute__((always_inline)) {
            store_pend(std::integral_constant<int, s0 + decltype(si)::value>{}, fast);
          });
        });
#pragma unroll
        for (int bi = 0; bi < PB; ++bi)
#pragma unroll
          for (int kb = 0; kb < 4; ++kb) pend[bi][kb] = acc[bi][kb];
        have_pend = true;
        pbase = ((n * K + j) * P + p0) * Q + q0 + 4 * gq;
        pcol = q0 + 4 * gq;
        ppart = decltype(part)::value;
      });
      copy_phase();
      gload(T + 2 * G);  // in flight during the next tile's MFMAs (nothing past the last tile)
    }
    // the last part's stores not issued during the last copies
    static_for<NST - NST_COPY>([&](auto si) __attribute__((always_inline)) {
      store_pend(std::integral_constant<int, NST_COPY + decltype(si)::value>{}, fast);
    });
  };
  if constexpr (OUTB && !PAIRED) {
    run(std::false_type{});
  } else {
    if (OUTB ? pair_out : vec_out)
      run(std::true_type{});
    else
      run(std::false_type{});
  }
}

// ---------------------------------------------------------------------------
// Pointwise (1x1) streaming kernels.
//
// With R = S = 1 the convolution is Out[n][k][px] = sum_c Ker[k][c] In[n][c][px]
// over the flattened pixels px of each image.  Each workgroup keeps its
// 64-row slice of Ker resident in LDS as rows [k][c] with a pitch of one float
// more than the stored channel count: lane (i, gq) reads row kb*16 + i at
// channel 4q + gq for the A operands, 16 distinct banks per 16-lane group.
// Each wave owns a contiguous range of `wpx` pixels (blocks of 16) and
// streams its In columns straight from HBM into a ring of registers with
// branch-free raw buffer loads: masked lanes start at 2^31, past the buffer's
// range, and read zeros.  No LDS traffic or barriers for In.  Both kernels
// require C % 4 == 0 and In below 1 GB (32-bit byte offsets).

// Fully unrolled kernel for a compile-time channel count C = 4 * NQ.
//
// Pixels go in units of 16: a wave with U units does U/2 blocks of 32 on
// v_mfma_f32_32x32x2f32 (two 32-row k blocks, two channels per MFMA) and,
// for odd U, one block of 16 on v_mfma_f32_16x16x4f32 (four 16-row k blocks,
// four channels).  Most of the work thus runs on the wider instruction: it
// reads half the operand registers per flop, and its accumulators can be
// reused every few instructions without stalls, while the pixel count per
// wave stays a multiple of 16.
//
// Each SIMD owns a contiguous range of `wpx` pixels.  With UB == 0 one wave
// per SIMD takes it (UA units).  With UB > 0 two waves share the SIMD: wave
// s takes the first 16 * UA pixels and wave s + 4 the next 16 * UB.  The two
// interleave their MFMAs, and when UB < UA the narrower wave ends first, so
// its stores drain while the other still computes.
//
// One step of the unrolled loop is one channel quad.  The Ker slice arrives
// in chunks of 64 channels straight to LDS (buffer loads with the LDS bit);
// chunk c+1 is requested during chunk c, so only the first chunk's latency
// precedes the first MFMA.
//
// Lane layouts (l = lane): 32x32x2 A[i][k] = lane (i = l%32, k = l/32), B[k][j]
// = lane (j = l%32, k = l/32), accumulator register v = (i = 8*(v/4) +
// 4*(l/32) + v%4, j = l%32); 16x16x4 A (i = l%16, k = l/16), B (j = l%16,
// k = l/16), register v = (i = 4*(l/16) + v, j = l%16).
template <int UA, int UB, int D, int NQ>
__global__ void __launch_bounds__(UB > 0 ? 512 : 256)
conv1x1_stream_kernel(const float* __restrict__ In, const float* __restrict__ Ker,
                      float* __restrict__ Out, const Geom g) {
  static_assert(NQ % 16 == 0, "Ker arrives in chunks of 16 channel quads");
  static_assert(UA >= 1 && UB >= 0, "pixel units per wave");
  constexpr int NW = UB > 0 ? 8 : 4;       // waves per workgroup
  constexpr int PITCH = 4 * NQ + 1;        // LDS Ker row pitch, floats
  constexpr int NCH = NQ / 16;             // Ker chunks of 64 channels
  extern __shared__ __align__(16) float lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int simd = wave & 3;
  const int l32 = lane & 31, h32 = lane >> 5;  // 32x32x2 lane coordinates
  const int l16 = lane & 15, h16 = lane >> 4;  // 16x16x4 lane coordinates
  const int C = g.C, K = g.K;
  const int HW = g.W;                   // kernel view: one row of H*W pixels per image
  const int total_px = g.N * HW;
  const int kt = blockIdx.x % g.tiles_k;
  const int pg = blockIdx.x / g.tiles_k;
  const int k0 = kt * 64;
  const int wpx = g.tw;                 // pixels per SIMD
  const int simd_begin = (pg * 4 + simd) * wpx;
  const int simd_end = min(simd_begin + wpx, total_px);

  // Ker chunk ch -> LDS: the NW waves copy 64 / NW rows each, 64 channels per
  // load (rows past K read zeros).
  const v4i krsrc = make_rsrc(Ker, g.ker_bytes);
  const unsigned lbase = (unsigned)(size_t)(lds_float*)lds;
  auto ker_chunk = [&](int ch) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 64 / NW; ++i) {
      const int kl = wave * (64 / NW) + i, k = k0 + kl;
      const unsigned voff = k < K ? (unsigned)(k * C + ch * 64 + lane) * 4u : kOob;
      dma_load<1>(krsrc, __builtin_amdgcn_readfirstlane(lbase + (unsigned)(kl * PITCH + ch * 64) * 4u), voff);
    }
  };
  __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(In), (short)0, (int)g.in_bytes, 0x00020000);
  const unsigned cstride = 4u * (unsigned)HW;  // bytes between channels

  // The work of one wave: U units of 16 pixels from px_begin (masked at px_end).
  auto body = [&](auto u_c, int px_begin, int px_end) __attribute__((always_inline)) {
    constexpr int U = decltype(u_c)::value;
    constexpr int NB32 = U / 2, NS16 = U % 2;
    constexpr int LPQ = 2 * NB32 + NS16;   // In loads per channel quad
    constexpr int LEAD = (48 / LPQ) < 16 ? (48 / LPQ) : 16;  // steps from a chunk's request to its wait
    static_assert(D >= 1 && D * LPQ <= 48 && D <= NQ && LEAD >= 1, "loads in flight stay within vmcnt");
    // In through raw buffer loads; masked lanes start at 2^31 and read zeros.
    auto in_off = [&](int px, int c) __attribute__((always_inline)) {
      const int n = px / HW, hw = px - n * HW;
      return (px < px_end) ? (unsigned)((n * C + c) * HW + hw) * 4u : kOob;
    };
    unsigned off32[NB32 > 0 ? NB32 : 1], off16 = 0;
#pragma unroll
    for (int b = 0; b < NB32; ++b) off32[b] = in_off(px_begin + 32 * b + l32, h32);
    if constexpr (NS16 > 0) off16 = in_off(px_begin + 32 * NB32 + l16, h16);
    float ring32[D][2][NB32 > 0 ? NB32 : 1], ring16[D];
    auto load = [&](int q) __attribute__((always_inline)) {
#pragma unroll
      for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int b = 0; b < NB32; ++b)
          ring32[q % D][e][b] = __builtin_bit_cast(
              float, __builtin_amdgcn_raw_buffer_load_b32(rsrc, off32[b] + (unsigned)(4 * q + 2 * e) * cstride, 0, 0));
      if constexpr (NS16 > 0)
        ring16[q % D] = __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(rsrc, off16 + (unsigned)(4 * q) * cstride, 0, 0));
    };
    // A operands, read one quad ahead: a32[e][kb] = Ker[k0 + 32kb + l32][4q + 2e + h32],
    // a16[kb] = Ker[k0 + 16kb + l16][4q + h16]
    const float* arow32 = lds + l32 * PITCH + h32;
    const float* arow16 = lds + l16 * PITCH + h16;
    float a32[2][2][2], a16[2][4];
    auto read_a = [&](int q, int buf) __attribute__((always_inline)) {
      if constexpr (NB32 > 0) {
#pragma unroll
        for (int e = 0; e < 2; ++e)
#pragma unroll
          for (int kb = 0; kb < 2; ++kb) a32[buf][e][kb] = arow32[kb * 32 * PITCH + 4 * q + 2 * e];
      }
      if constexpr (NS16 > 0) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) a16[buf][kb] = arow16[kb * 16 * PITCH + 4 * q];
      }
    };
    v16f acc32[NB32 > 0 ? NB32 : 1][2];
    v4f acc16[4];
#pragma unroll
    for (int b = 0; b < NB32; ++b)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) acc32[b][kb] = v16f{};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) acc16[kb] = v4f{0.f, 0.f, 0.f, 0.f};

    // prologue: first Ker chunk, then the ring, then wait for the chunk (the
    // ring's D * LPQ loads are younger and may stay in flight)
    ker_chunk(0);
#pragma unroll
    for (int q = 0; q < D; ++q) load(q);
    wait_vmcnt_opaque<D * LPQ>();
    __syncthreads();
    read_a(0, 0);
    static_for<NQ>([&](auto q_c) __attribute__((always_inline)) {
      constexpr int q = decltype(q_c)::value;
      constexpr int buf = q & 1;
      constexpr bool chunk_end = q % 16 == 15 && q / 16 + 1 < NCH;
      if constexpr (q + 1 < NQ && !chunk_end) read_a(q + 1, buf ^ 1);
      __builtin_amdgcn_sched_barrier(0);  // issue the A reads first
      if constexpr (q % 16 == 16 - LEAD && q / 16 + 1 < NCH) ker_chunk(q / 16 + 1);
#pragma unroll
      for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int b = 0; b < NB32; ++b)
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
            acc32[b][kb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a32[buf][e][kb], ring32[q % D][e][b],
                                                                acc32[b][kb], 0, 0, 0);
      if constexpr (NS16 > 0) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
          acc16[kb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a16[buf][kb], ring16[q % D], acc16[kb], 0, 0, 0);
      }
      if constexpr (q + D < NQ) load(q + D);
      if constexpr (chunk_end) {
        // the next chunk was requested LEAD steps ago; LEAD * LPQ ring loads are younger
        wait_vmcnt_opaque<LEAD * LPQ>();
        __syncthreads();
        read_a(q + 1, buf ^ 1);
      }
      // keep each refill right behind the MFMAs that free its slot: left
      // alone, the scheduler sinks loads towards their uses and the ring
      // degenerates to a few loads in flight
      __builtin_amdgcn_sched_barrier(0);
    });

    // stores: 32 consecutive pixels (two rows of k) or 16 (four rows) per
    // instruction, with the non-temporal hint (Out is not read back here;
    // measured about 3% faster on the 56x56 layer)
#pragma unroll
    for (int b = 0; b < NB32; ++b) {
      const int px = px_begin + 32 * b + l32;
      if (px < px_end) {
        const int n = px / HW, hw = px - n * HW;
        float* ob = Out + (size_t)n * K * HW + hw;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int k = k0 + 32 * kb + 8 * (v / 4) + 4 * h32 + v % 4;
            if (k < K) __builtin_nontemporal_store(acc32[b][kb][v], &ob[(size_t)k * HW]);
          }
      }
    }
    if constexpr (NS16 > 0) {
      const int px = px_begin + 32 * NB32 + l16;
      if (px < px_end) {
        const int n = px / HW, hw = px - n * HW;
        float* ob = Out + (size_t)n * K * HW + hw;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int k = k0 + 16 * kb + 4 * h16 + v;
            if (k < K) __builtin_nontemporal_store(acc16[kb][v], &ob[(size_t)k * HW]);
          }
      }
    }
  };
  if constexpr (UB > 0) {
    if (wave >= 4) {
      body(std::integral_constant<int, UB>{}, simd_begin + 16 * UA, simd_end);
      return;
    }
  }
  body(std::integral_constant<int, UA>{}, simd_begin, min(simd_begin + 16 * UA, simd_end));
}

// Balanced pointwise kernel for a compile-time channel count C = 4 * NQ.
//
// The unrolled kernel above gives each SIMD a whole number of 16-pixel
// units, so a pixel count that is not a multiple of 16 x 4 x 256 leaves CUs
// idle or SIMDs uneven (the 1x1 N=32 C=256 56x56 layer: 7 units on each of
// 896 SIMDs, 32 CUs idle).  Here every workgroup (four waves, one per SIMD)
// does the same work: NB blocks of 128 pixels and a 16-pixel tail block.
// With tile_cols = PW = 128 * NB + T (0 < T <= 16), the grid has
// G = ceil(pixels / PW) workgroups per k tile, and workgroup p takes
// 128-pixel block j at pixel (j G + p) 128 and the tail at NB G 128 + 16 p
// (tail pixels past the end masked).  Blocks are handed out in grid stride,
// so at any time the grid reads, and writes, one compact window of every
// channel row rather than G scattered ones, and every block starts on a
// 512-byte boundary (measured on the 1x1 N=32 C=256 layer: 4% faster than
// contiguous shares; strided 1x1 N=32 C=64: 11%):
//   * wave s computes the NB 32-pixel blocks at (j G + p) 128 + 32 s,
//     j = 0 .. NB-1, one after another (so the four waves read adjacent
//     128-byte pieces of each channel row).  Each block accumulates over all
//     C channels, the even and odd channel pairs of each quad in separate
//     accumulators (four independent 32x32x2 chains keep the MFMA pipe full
//     with one wave per SIMD); the two are added and the block's 32 results
//     are stored over the steps of the next block, which spreads the Out
//     writes over the whole kernel instead of one burst per block (the last
//     block stores at the end);
//   * the 16-pixel tail block (masked past the last pixel) has its 64 rows
//     of k split among the four waves, 16 rows each on one 16x16x4
//     accumulator, computed alongside each wave's last block.  The blocks
//     cover NB G 128 pixels and the tails 16 G more, at least all of them
//     since G PW >= pixels.
// In streams from HBM into a ring of registers D steps ahead (branch-free
// raw buffer loads, masked lanes read zeros past the buffer's range).  Ker
// (64 rows of this k tile, all C channels) is staged through registers into
// LDS in chunks of 64 channels during the first block, each chunk requested
// a whole chunk ahead; every load is visible to the compiler, so its waits
// are exact.  Strided or padded 1x1 layers read In through the phase
// mapping (no separate pass).  Requires C % 64 == 0, In below 1 GB and Out
// below 2 GB (32-bit offsets).
template <int NB, int D, int NQ>
__global__ void __launch_bounds__(256)
conv1x1_bal_kernel(const float* __restrict__ In, const float* __restrict__ Ker, float* __restrict__ Out,
                   const Geom g) {
  static_assert(NQ % 16 == 0, "Ker arrives in chunks of 16 channel quads");
  static_assert(NB >= 1 && D >= 2 && 3 * D <= 60, "ring loads in flight stay within vmcnt");
  constexpr int PITCH = 4 * NQ + 1;  // LDS Ker row pitch, floats
  constexpr int NCH = NQ / 16;       // Ker chunks of 64 channels
  constexpr int NSTEP = NB * NQ;     // one step = one channel quad of one block
  extern __shared__ __align__(16) float lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, h32 = lane >> 5;  // 32x32x2 lane coordinates
  const int l16 = lane & 15, h16 = lane >> 4;  // 16x16x4 lane coordinates
  const int C = g.C, K = g.K;
  const int HW = g.W;  // kernel view: one row of H*W pixels per image
  const int total_px = g.N * HW;
  const int kt = blockIdx.x % g.tiles_k;
  const int pg = blockIdx.x / g.tiles_k;
  const int k0 = kt * 64;
  const int GP = g.tiles_rows;  // workgroups per k tile
  const int Pend = total_px;
  const int ptail = NB * GP * 128 + 16 * pg;
  // first pixel of this wave's 32 in 128-pixel block j
  auto bpx = [&](int j) __attribute__((always_inline)) { return (j * GP + pg) * 128 + 32 * wave; };

  __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(In), (short)0, (int)g.in_bytes, 0x00020000);
  __amdgpu_buffer_rsrc_t krsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(Ker), (short)0, (int)g.ker_bytes, 0x00020000);
  // Strided or padded 1x1 layers (conv_fwd_ex, g.nph = 1) read the
  // caller's In through the phase mapping: inner pixel (yi, xi) of image n
  // is In pixel (yi sh - ph, xi sw - pw), zero outside the image.
  const unsigned cstride = 4u * (unsigned)(g.nph ? g.H0 * g.W0 : HW);  // bytes between channels
  auto in_off = [&](int px, int c) __attribute__((always_inline)) {
    const int n = px / HW, hw = px - n * HW;
    if (px >= Pend) return kOob;
    if (g.nph == 0) return (unsigned)((n * C + c) * HW + hw) * 4u;
    const int yi = fdiv(hw, g.dv_Wi), xi = hw - yi * g.Wi;
    const int iy = yi * g.sh - g.ph, ix = xi * g.sw - g.pw;
    if (iy < 0 || iy >= g.H0 || ix < 0 || ix >= g.W0) return kOob;
    return (unsigned)(((n * g.C0 + c) * g.H0 + iy) * g.W0 + ix) * 4u;
  };
  unsigned off32[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) off32[j] = in_off(bpx(j) + l32, h32);
  const unsigned off16 = in_off(ptail + l16, h16);

  // Ker chunk ch: 64 rows x 64 channels; lane (wave, i, lane) holds row
  // 16 * wave + 4 * i + lane / 16, channels 4 * (lane % 16) .. + 3.
  v4f kst[4];
  auto ker_load = [&](int ch) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = k0 + 16 * wave + 4 * i + (lane >> 4);
      const unsigned voff = k < K ? (unsigned)(k * C + ch * 64 + 4 * (lane & 15)) * 4u : kOob;
      kst[i] = __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(krsrc, voff, 0, 0));
    }
  };
  auto ker_store = [&](int ch) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float* row = lds + (16 * wave + 4 * i + (lane >> 4)) * PITCH + ch * 64 + 4 * (lane & 15);
#pragma unroll
      for (int e = 0; e < 4; ++e) row[e] = kst[i][e];
    }
  };

  // ring slot of step t: two 32x32x2 B operands (channel pairs e = 0, 1 of
  // the quad) and, in the last block, the tail block's 16x16x4 B operand
  float ring32[D][2], ring16[D];
  auto load = [&](auto t_c) __attribute__((always_inline)) {
    constexpr int t = decltype(t_c)::value;
    constexpr int j = t / NQ, q = t % NQ;
#pragma unroll
    for (int e = 0; e < 2; ++e)
      ring32[t % D][e] = __builtin_bit_cast(
          float, __builtin_amdgcn_raw_buffer_load_b32(rsrc, off32[j] + (unsigned)(4 * q + 2 * e) * cstride, 0, 0));
    if constexpr (j == NB - 1)
      ring16[t % D] = __builtin_bit_cast(
          float, __builtin_amdgcn_raw_buffer_load_b32(rsrc, off16 + (unsigned)(4 * q) * cstride, 0, 0));
  };
  // A operands of quad q, read one step ahead: a32[e][kb] = Ker[k0 + 32 kb + l32][4q + 2e + h32],
  // a16 = Ker[k0 + 16 wave + l16][4q + h16]
  const float* arow32 = lds + l32 * PITCH + h32;
  const float* arow16 = lds + (16 * wave + l16) * PITCH + h16;
  float a32[2][2][2], a16[2];
  auto read_a = [&](int q, int buf, bool tail) __attribute__((always_inline)) {
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) a32[buf][e][kb] = arow32[kb * 32 * PITCH + 4 * q + 2 * e];
    if (tail) a16[buf] = arow16[4 * q];
  };
  v16f acc[2][2];  // [kb][e]
  v4f acc16 = v4f{0.f, 0.f, 0.f, 0.f};
  // A finished block's 32 results (every block but the last) are stored
  // over the steps of the next block, results 32 q / NQ .. 32 (q + 1) / NQ - 1
  // at step q (one every NQ / 32 steps, or 32 / NQ per step).  Stores and loads
  // share one completion counter, so ring loads issued behind a burst of 32
  // stores (32 KB per CU, draining at the CU's share of the HBM write rate)
  // would wait for all of them and stall the next block.  32-bit offsets
  // (Out below 2 GB); a masked lane's offset is past the buffer's range.
  const __amdgpu_buffer_rsrc_t orsrc = __builtin_amdgcn_make_buffer_rsrc(
      Out, (short)0, (int)((unsigned)g.N * (unsigned)K * (unsigned)HW * 4u), 0x00020000);
  float pend[32];
  unsigned pend_base = kOob;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int e = 0; e < 2; ++e) acc[kb][e] = v16f{};

  // prologue: Ker chunk 0, the ring, then chunk 0 into LDS
  ker_load(0);
  static_for<D>([&](auto t_c) __attribute__((always_inline)) { load(t_c); });
  ker_store(0);
  if constexpr (NCH > 1) ker_load(1);
  __syncthreads();
  read_a(0, 0, NB == 1);

  static_for<NSTEP>([&](auto t_c) __attribute__((always_inline)) {
    constexpr int t = decltype(t_c)::value;
    constexpr int j = t / NQ, q = t % NQ;
    constexpr int buf = t & 1;
    constexpr bool tail = j == NB - 1;
    // end of a Ker chunk during the first block: the next chunk (requested
    // a chunk ago) goes to LDS before its first A read
    constexpr bool chunk_end = j == 0 && q % 16 == 15 && q / 16 + 1 < NCH;
    constexpr int tn = t + 1;
    if constexpr (tn < NSTEP && !chunk_end) read_a(tn % NQ, buf ^ 1, tn / NQ == NB - 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        acc[kb][e] = __builtin_amdgcn_mfma_f32_32x32x2f32(a32[buf][e][kb], ring32[t % D][e], acc[kb][e], 0, 0, 0);
    if constexpr (tail) acc16 = __builtin_amdgcn_mfma_f32_16x16x4f32(a16[buf], ring16[t % D], acc16, 0, 0, 0);
    if constexpr (t + D < NSTEP) load(std::integral_constant<int, t + D>{});
    if constexpr (j >= 1) {
      // the previous block's results r: row 32 kb + 8 (v / 4) + 4 h32 + v % 4
      static_for<(32 * (q + 1)) / NQ - (32 * q) / NQ>([&](auto i_c) __attribute__((always_inline)) {
        constexpr int r = (32 * q) / NQ + decltype(i_c)::value;
        constexpr int kb = r / 16, v = r % 16;
        const int k = k0 + 32 * kb + 8 * (v / 4) + 4 * h32 + v % 4;
        const float val = pend[r];
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, val), orsrc,
                                              k < K ? pend_base + (unsigned)(k * HW) * 4u : kOob, 0, kStoreNT);
      });
    }
    if constexpr (chunk_end) {
      ker_store(q / 16 + 1);
      if constexpr (q / 16 + 2 < NCH) ker_load(q / 16 + 2);
      __syncthreads();
      read_a(tn % NQ, buf ^ 1, tn / NQ == NB - 1);
    }
    if constexpr (q == NQ - 1 && j < NB - 1) {
      // block j done: add the two channel-pair halves into the pending
      // results, then restart
      const int px = bpx(j) + l32;
      const int n = px / HW, hw = px - n * HW;
      pend_base = px < Pend ? (unsigned)(n * K * HW + hw) * 4u : kOob;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) pend[16 * kb + v] = acc[kb][0][v] + acc[kb][1][v];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 2; ++e) acc[kb][e] = v16f{};
    }
    if constexpr (q == NQ - 1 && j == NB - 1) {
      // last block done: add the two channel-pair halves and store 32 pixels
      // (two rows of k per instruction, streaming hint)
      const int px = bpx(j) + l32;
      if (px < Pend) {
        const int n = px / HW, hw = px - n * HW;
        float* ob = Out + (size_t)n * K * HW + hw;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int k = k0 + 32 * kb + 8 * (v / 4) + 4 * h32 + v % 4;
            if (k < K) __builtin_nontemporal_store(acc[kb][0][v] + acc[kb][1][v], &ob[(size_t)k * HW]);
          }
      }
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 2; ++e) acc[kb][e] = v16f{};
    }
    // keep each refill right behind the MFMAs that free its slot
    __builtin_amdgcn_sched_barrier(0);
  });
  // the tail block's 16 rows of k owned by this wave
  const int px = ptail + l16;
  if (px < Pend) {
    const int n = px / HW, hw = px - n * HW;
    float* ob = Out + (size_t)n * K * HW + hw;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int k = k0 + 16 * wave + 4 * h16 + v;
      if (k < K) __builtin_nontemporal_store(acc16[v], &ob[(size_t)k * HW]);
    }
  }
}

// Looped kernel for any channel count (C % 4 == 0): D quads per loop trip,
// the Ker slice zero-padded to whole trips and copied to LDS up front; two
// phases of NB1 and NB2 pixel blocks.
template <int NB1, int NB2, int D>
__global__ void __launch_bounds__(kThreads)
conv1x1_stream_loop_kernel(const float* __restrict__ In, const float* __restrict__ Ker,
                           float* __restrict__ Out, const Geom g) {
  static_assert(NB1 > 0 && D % 2 == 0, "phase one is not empty; the A double buffer alternates");
  extern __shared__ __align__(16) float lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int j = lane & 15, gq = lane >> 4;
  const int C = g.C, K = g.K;
  const int HW = g.W;
  const int total_px = g.N * HW;
  const int kt = blockIdx.x % g.tiles_k;
  const int pg = blockIdx.x / g.tiles_k;
  const int k0 = kt * 64;
  const int wpx = g.tw;
  const int px_begin = (pg * 4 + wave) * wpx;
  const int px_end = min(px_begin + wpx, total_px);
  const int nq = C / 4;
  const int nq_pad = (nq + D - 1) / D * D;
  const int cpad = nq_pad * 4, pitch = cpad + 1;

  // Ker slice -> LDS rows [k][c]: batches of coalesced loads, all in flight
  // before any is waited on.
  {
    constexpr int FB = 16;
    for (int e0 = 0; e0 < 64 * cpad; e0 += kThreads * FB) {
      float kv[FB];
#pragma unroll
      for (int i = 0; i < FB; ++i) {
        const int e = e0 + tid + i * kThreads;
        const int kl = e / cpad, c = e - kl * cpad;
        const int k = k0 + kl;
        kv[i] = (e < 64 * cpad && k < K && c < C) ? Ker[(size_t)k * C + c] : 0.f;
      }
#pragma unroll
      for (int i = 0; i < FB; ++i) {
        const int e = e0 + tid + i * kThreads;
        const int kl = e / cpad, c = e - kl * cpad;
        if (e < 64 * cpad) lds[kl * pitch + c] = kv[i];
      }
    }
  }
  __syncthreads();
  __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(In), (short)0, (int)g.in_bytes, 0x00020000);
  const unsigned qstride = 16u * (unsigned)HW;

  auto phase = [&](auto nb_const, int blk0) {
    constexpr int NB = decltype(nb_const)::value;
    if constexpr (NB > 0) {
      unsigned voff[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int px = px_begin + (blk0 + b) * 16 + j;
        const int n = px / HW, hw = px - n * HW;
        voff[b] = (px < px_end) ? (unsigned)((n * C + gq) * HW + hw) * 4u : kOob;
      }
      v4f acc[4][NB];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int b = 0; b < NB; ++b) acc[kb][b] = v4f{0.f, 0.f, 0.f, 0.f};
      float ring[D][NB];
      // quads past the channel range add 2^30 (wave-uniform): with In below
      // 1 GB both sentinels land past the buffer's range without wrapping
      auto load = [&](int q, int slot) {
        const unsigned qoff = (unsigned)q * qstride + (q < nq ? 0u : 0x40000000u);
#pragma unroll
        for (int b = 0; b < NB; ++b)
          ring[slot][b] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc, voff[b] + qoff, 0, 0));
      };
#pragma unroll
      for (int d = 0; d < D; ++d) load(d, d);
      const float* arow = lds + j * pitch + gq;
      float a[2][4];
      auto read_a = [&](int q, float* dst) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) dst[kb] = arow[kb * 16 * pitch + 4 * q];
      };
      read_a(0, a[0]);
      for (int q0 = 0; q0 < nq_pad; q0 += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
          read_a(min(q0 + d + 1, nq_pad - 1), a[(d + 1) & 1]);  // the last one is unused
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int b = 0; b < NB; ++b)
              acc[kb][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[d & 1][kb], ring[d][b], acc[kb][b], 0, 0, 0);
          load(q0 + d + D, d);  // past the last quad this reads zeros
          __builtin_amdgcn_sched_barrier(0);
        }
      }
#pragma unroll
      for (int b = 0; b < NB; ++b) {  // non-temporal stores, as in the unrolled kernel
        const int px = px_begin + (blk0 + b) * 16 + j;
        if (px < px_end) {
          const int n = px / HW, hw = px - n * HW;
          float* ob = Out + (size_t)n * K * HW + hw;
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const int k = k0 + kb * 16 + 4 * gq + v;
              if (k < K) __builtin_nontemporal_store(acc[kb][b][v], &ob[(size_t)k * HW]);
            }
        }
      }
    }
  };
  phase(std::integral_constant<int, NB1>{}, 0);
  phase(std::integral_constant<int, NB2>{}, NB1);
}

typedef void (*KernelF32)(const float*, const float*, float*, const Geom);
typedef void (*KernelBF16)(const unsigned short*, const unsigned short*, float*, const Geom);

struct Instance {
  Variant v;
  KernelF32 f32;
  KernelBF16 bf16;
  KernelBF16 bf16_outb;  // the same kernel writing bf16 Out (transposing bf16 family only)
};

// ---------------------------------------------------------------------------
// Second pass of a split reduction: Out[i] = W[0][i] + W[1][i] + ... over the
// split channel ranges' partial outputs, always in range order, so the result
// does not depend on which workgroup finished first.  VEC4: n % 4 == 0 and a
// 16-byte aligned Out (the workspace always is).
template <bool VEC4>
__global__ void __launch_bounds__(256)
splitk_reduce_kernel(const float* __restrict__ W, float* __restrict__ Out, int64_t n, int split) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  if constexpr (VEC4) {
    const int64_t n4 = n / 4;
    const v4f* W4 = reinterpret_cast<const v4f*>(W);
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride) {
      v4f acc = W4[i];
      for (int r = 1; r < split; ++r) acc += W4[(size_t)r * n4 + i];
      reinterpret_cast<v4f*>(Out)[i] = acc;
    }
  } else {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) {
      float acc = W[i];
      for (int r = 1; r < split; ++r) acc += W[(size_t)r * n + i];
      Out[i] = acc;
    }
  }
}

// ---------------------------------------------------------------------------
// Strided, zero-padded convolution as a stride-1 valid one (polyphase or
// space-to-depth rewrite).  With input row y = h*sh + r - ph, write the tap
// r = sh*r' + a (a < sh): the row becomes sh*(h + r') + (a - ph), so phase
// image a of the padded input, X_a[y'] = X[sh*y' + a - ph], is read at
// h + r' -- a stride-1 correlation over r'.  Likewise for columns.  The
// phases (a, b) become extra input channels, (c*na + a)*nb + b, with na =
// min(sh, R) and nb = min(sw, S) (phases no tap reaches are left out), and
// the kernel gets taps r' < ceil(R/sh), t' < ceil(S/sw), zero where
// sh*r' + a >= R or sw*t' + b >= S.

// Inp[n][(c*na + a)*nb + b][y][x] = In[n][c][y*sh + a - ph][x*sw + b - pw],
// zero outside the input.  One element per thread, grid-stride; 32-bit
// index arithmetic (both tensors hold fewer than 2^31 elements).
template <typename T>
__global__ void __launch_bounds__(256)
phase_split_kernel(const T* __restrict__ In, T* __restrict__ Inp, PhaseGeom p) {
  const int Cp = p.C * p.na * p.nb;
  const int total = p.N * Cp * p.Hp * p.Wp;
  for (int i = blockIdx.x * 256 + threadIdx.x; i < total; i += gridDim.x * 256) {
    int t = i;
    const int x = t % p.Wp;
    t /= p.Wp;
    const int y = t % p.Hp;
    t /= p.Hp;
    const int cp = t % Cp;
    const int n = t / Cp;
    const int b = cp % p.nb, a = (cp / p.nb) % p.na, c = cp / (p.na * p.nb);
    const int iy = y * p.sh + a - p.ph, ix = x * p.sw + b - p.pw;
    Inp[i] = (iy >= 0 && iy < p.H && ix >= 0 && ix < p.W) ? In[((n * p.C + c) * p.H + iy) * p.W + ix] : T(0);
  }
}

// Kp[k][(c*na + a)*nb + b][r'][t'] = Ker[k][c][r'*sh + a][t'*sw + b], zero
// past the R x S taps.
template <typename T>
__global__ void __launch_bounds__(256)
ker_phase_kernel(const T* __restrict__ Ker, T* __restrict__ Kp, PhaseGeom p) {
  // Ker and Kp hold fewer than 2^31 elements (checked on the host), so the
  // index math is 32-bit (64-bit divisions measured about 15% slower).
  const unsigned Cp = (unsigned)(p.C * p.na * p.nb);
  const unsigned Rp = (unsigned)p.Rp, Sp = (unsigned)p.Sp, nb = (unsigned)p.nb, na = (unsigned)p.na;
  const unsigned total = (unsigned)p.K * Cp * Rp * Sp;
  for (unsigned i = blockIdx.x * 256u + threadIdx.x; i < total; i += gridDim.x * 256u) {
    unsigned t = i;
    const unsigned tt = t % Sp; t /= Sp;
    const unsigned rr = t % Rp; t /= Rp;
    const unsigned cp = t % Cp;
    const unsigned k = t / Cp;
    const unsigned b = cp % nb, a = (cp / nb) % na, c = cp / (na * nb);
    const int r = (int)(rr * p.sh + a), s = (int)(tt * p.sw + b);
    Kp[i] = (r < p.R && s < p.S) ? Ker[((k * (unsigned)p.C + c) * (unsigned)p.R + r) * (unsigned)p.S + s] : T(0);
  }
}

// Out (bf16) = fp32 partial result rounded to nearest even, for the bf16
// output of kernels that only write fp32.
__global__ void __launch_bounds__(256)
round_bf16_kernel(const float* __restrict__ src, unsigned short* __restrict__ dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    dst[i] = __builtin_bit_cast(unsigned short, (__bf16)src[i]);
}

// fp32 = the bf16 value (exact: the bf16 bits are the high half).
__global__ void __launch_bounds__(256)
widen_bf16_kernel(const unsigned short* __restrict__ src, float* __restrict__ dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    dst[i] = __builtin_bit_cast(float, (unsigned)src[i] << 16);
}

#define F32_INST(ID, WK, WP, TC, RC, SC, MAXNI, MAXNK, KV)                                  \
  Instance{Variant{ID, CONV_DTYPE_F32, FAMILY_STAGED, WK, WP, TC, RC, SC, MAXNI, MAXNK, KV, 1, \
                   kThreads, 2},                                                             \
           &conv_f32_kernel<WK, WP, TC, RC, SC, MAXNI, MAXNK, KV>, nullptr}

#define F32_DMA(ID, WK, WP, NW, TC, RC, SC, NS, NLI, KVI, NLK, KVK)                              \
  Instance{Variant{ID, CONV_DTYPE_F32, FAMILY_DMA, WK, WP, TC, RC, SC, NLI, NLK, KVK, KVI, NW * 64, \
                   NS, 0},                                                                       \
           &conv_f32_dma_kernel<WK, WP, NW, TC, RC, SC, NS, NLI, KVI, NLK, KVK>, nullptr}

// the same pipeline with NWC channel groups of waves (16x16x4 loop)
#define F32_DMA_CG(ID, WK, WP, NW, NWC, TC, RC, SC, NS, NLI, KVI, NLK, KVK)                      \
  Instance{Variant{ID, CONV_DTYPE_F32, FAMILY_DMA, WK, WP, TC, RC, SC, NLI, NLK, KVK, KVI, NW * 64, \
                   NS, 0, NWC},                                                                  \
           &conv_f32_dma_kernel<WK, WP, NW, TC, RC, SC, NS, NLI, KVI, NLK, KVK, false, NWC>, nullptr}

// the same pipeline skipping the zero taps of a stride-2 odd-tap layer's
// phases (conv_fwd_ex only)
#define F32_DMA_PS(ID, WK, WP, NW, TC, RC, SC, NS, NLI, KVI, NLK, KVK)                           \
  Instance{Variant{ID, CONV_DTYPE_F32, FAMILY_DMA, WK, WP, TC, RC, SC, NLI, NLK, KVK, KVI, NW * 64, \
                   NS, 0, 1, 1},                                                                 \
           &conv_f32_dma_kernel<WK, WP, NW, TC, RC, SC, NS, NLI, KVI, NLK, KVK, false, 1, true>, nullptr}

// the same pipeline with the 32x32x2 inner loop (WK = 4, WP even)
#define F32_DMA32(ID, WP, NW, TC, RC, SC, NS, NLI, KVI, NLK, KVK)                                \
  Instance{Variant{ID, CONV_DTYPE_F32, FAMILY_DMA, 4, WP, TC, RC, SC, NLI, NLK, KVK, KVI, NW * 64, \
                   NS, 1},                                                                       \
           &conv_f32_dma_kernel<4, WP, NW, TC, RC, SC, NS, NLI, KVI, NLK, KVK, true>, nullptr}

#define F32_STREAM1X1(ID, UA, UB, D, NQ)                                                   \
  Instance{Variant{ID, CONV_DTYPE_F32, FAMILY_STREAM1X1, 4, UA + UB, 4 * NQ, 1, 1, UA, UB, 1, 1, \
                   (UB > 0 ? 512 : 256), D},                                                 \
           &conv1x1_stream_kernel<UA, UB, D, NQ>, nullptr}

#define F32_STREAM1X1_BAL(ID, NB, D, NQ)                                                     \
  Instance{Variant{ID, CONV_DTYPE_F32, FAMILY_STREAM1X1_BAL, 4, 2 * NB + 1, 4 * NQ, 1, 1, NB, 1, 4, 1, \
                   kThreads, D},                                                                 \
           &conv1x1_bal_kernel<NB, D, NQ>, nullptr}

#define F32_STREAM1X1_LOOP(ID, NB1, NB2, D)                                                  \
  Instance{Variant{ID, CONV_DTYPE_F32, FAMILY_STREAM1X1_LOOP, 4, NB1 + NB2, 0, 1, 1, NB1, NB2, \
                   1, 1, kThreads, D},                                                       \
           &conv1x1_stream_loop_kernel<NB1, NB2, D>, nullptr}

#define BF16_TR_INST(ID, TR, TW, RC, SC)                                                       \
  Instance{Variant{ID, CONV_DTYPE_BF16, FAMILY_BF16_TR, 4, TR * TW / 64, 32, RC, SC, TR, TW, 8, 1, \
                   kThreads, 1},                                                                  \
           nullptr, &conv_bf16_tr_kernel<TR, TW, RC, SC, false>,                                    \
           &conv_bf16_tr_kernel<TR, TW, RC, SC, true>}

#define BF16_INST(ID, WK, WP, RC, SC, MAXIT)                                                  \
  Instance{Variant{ID, CONV_DTYPE_BF16, FAMILY_BF16, WK, WP, 32, RC, SC, MAXIT, 0, 8, 8, kThreads, \
                   1},                                                                        \
           nullptr, &conv_bf16_kernel<WK, WP, RC, SC, MAXIT>}

const Instance kInstances[] = {
    // ---- pointwise streaming (Ker resident in LDS, In straight to registers)
    // unrolled for C = 4 * NQ: (16-pixel units of the first wave per SIMD,
    // of the second, ring depth in channel quads)
    F32_STREAM1X1(301, 4, 3, 6, 64),
    F32_STREAM1X1(302, 4, 3, 4, 64),
    F32_STREAM1X1(303, 7, 0, 4, 64),
    F32_STREAM1X1(304, 7, 0, 6, 64),
    F32_STREAM1X1(305, 4, 4, 6, 64),
    F32_STREAM1X1(306, 5, 2, 5, 64),
    F32_STREAM1X1(307, 4, 3, 6, 16),
    F32_STREAM1X1(308, 4, 3, 6, 32),
    F32_STREAM1X1(309, 4, 3, 6, 128),
    // any C % 4 == 0: (phase-1 blocks, phase-2 blocks, quads per trip)
    // balanced pointwise kernel: NB 32-pixel blocks per wave plus a k-split tail
    F32_STREAM1X1_BAL(321, 3, 16, 64),
    F32_STREAM1X1_BAL(322, 3, 12, 64),
    F32_STREAM1X1_BAL(323, 2, 16, 64),
    F32_STREAM1X1_BAL(324, 1, 16, 64),
    F32_STREAM1X1_BAL(325, 3, 16, 32),
    F32_STREAM1X1_BAL(326, 2, 16, 32),
    F32_STREAM1X1_BAL(327, 3, 16, 16),
    F32_STREAM1X1_BAL(328, 2, 16, 16),
    F32_STREAM1X1_BAL(329, 2, 16, 128),
    F32_STREAM1X1_BAL(330, 1, 16, 128),
    F32_STREAM1X1_BAL(331, 3, 16, 96),
    F32_STREAM1X1_BAL(332, 2, 16, 96),
    F32_STREAM1X1_LOOP(311, 4, 3, 8),
    F32_STREAM1X1_LOOP(312, 4, 0, 8),
    F32_STREAM1X1_LOOP(313, 2, 2, 8),
    F32_STREAM1X1_LOOP(314, 2, 0, 8),
    // ---- direct-to-LDS pipeline
    // 3x3 taps
    F32_DMA(101, 1, 13, 4, 8, 3, 3, 3, 9, 1, 5, 4),
    F32_DMA(102, 4, 4, 4, 8, 3, 3, 3, 12, 1, 10, 4),
    F32_DMA(103, 2, 2, 4, 8, 3, 3, 3, 8, 1, 5, 4),
    F32_DMA(104, 1, 4, 4, 8, 3, 3, 3, 8, 1, 5, 4),
    F32_DMA(105, 2, 4, 4, 8, 3, 3, 3, 12, 1, 5, 4),
    F32_DMA(106, 1, 7, 8, 8, 3, 3, 3, 5, 1, 3, 4),
    F32_DMA(107, 1, 4, 8, 8, 3, 3, 3, 4, 1, 3, 4),
    F32_DMA(108, 2, 4, 8, 8, 3, 3, 3, 6, 1, 3, 4),
    // 2x2 and 4x4 taps: stride-2 3x3 and 7x7 layers after the polyphase rewrite
    F32_DMA(109, 4, 4, 4, 8, 2, 2, 3, 12, 1, 5, 4),
    F32_DMA(110, 1, 7, 8, 8, 2, 2, 3, 5, 1, 2, 4),
    F32_DMA(111, 2, 4, 8, 8, 2, 2, 3, 6, 1, 2, 4),
    F32_DMA(112, 4, 4, 4, 8, 4, 4, 3, 14, 1, 8, 4),
    F32_DMA(113, 1, 7, 8, 8, 4, 4, 3, 6, 1, 5, 4),
    F32_DMA(114, 2, 4, 8, 8, 4, 4, 3, 7, 1, 5, 4),
    // 4x4 taps, four channels per step (the 7x7 stride-2 layer's 12 phase
    // channels in three whole steps); 2x2 taps, sixteen per step (more
    // MFMAs between barriers on deep channel ranges)
    F32_DMA(115, 1, 7, 8, 4, 4, 4, 2, 3, 1, 3, 4),
    F32_DMA(116, 2, 4, 8, 4, 4, 4, 2, 3, 1, 3, 4),
    F32_DMA(117, 4, 4, 4, 16, 2, 2, 3, 6, 1, 5, 4),
    F32_DMA(118, 2, 4, 8, 16, 2, 2, 3, 10, 1, 3, 4),
    // phase-skip twin of 118 for stride-2 3x3 layers (four input channels
    // per phase and step)
    F32_DMA_PS(192, 2, 4, 8, 16, 2, 2, 3, 10, 1, 3, 4),
    // squat wave tiles (4 k blocks x 4..8 pixel blocks), Ker rows loaded
    // element-wise so their LDS pitch can be conflict-free
    F32_DMA(141, 4, 4, 4, 8, 3, 3, 3, 7, 1, 19, 1),
    F32_DMA(142, 4, 4, 8, 8, 3, 3, 3, 4, 1, 10, 1),
    F32_DMA(143, 2, 4, 8, 8, 3, 3, 3, 4, 1, 10, 1),
    F32_DMA(144, 4, 2, 4, 8, 3, 3, 3, 4, 1, 19, 1),
    F32_DMA(145, 2, 8, 8, 8, 3, 3, 3, 7, 1, 10, 1),
    // few input channels (the first layer of a network): four per step,
    // 32-row k tiles
    F32_DMA(146, 2, 4, 8, 4, 3, 3, 3, 7, 1, 3, 1),
    F32_DMA(147, 2, 2, 4, 4, 3, 3, 3, 7, 1, 5, 1),
    // channel groups of waves (WK, WP, waves, groups, channels per step, ...):
    // small layers without a split reduction
    F32_DMA_CG(161, 2, 2, 4, 4, 16, 3, 3, 3, 7, 1, 5, 4),
    F32_DMA_CG(162, 2, 2, 8, 8, 32, 3, 3, 2, 7, 1, 5, 4),
    // the same with fewer In loads (tiles whose In halo fits): the small
    // 3x3 layers' plans issue no empty loads
    F32_DMA_CG(179, 2, 2, 8, 8, 32, 3, 3, 2, 4, 1, 5, 4),
    F32_DMA_CG(180, 2, 2, 4, 4, 16, 3, 3, 4, 4, 1, 5, 4),
    // 32 k x 7 blocks per wave, one wave per channel group: 32 x 98-pixel
    // tiles cover the 3x3 7x7 N32 layer in 256 workgroups with 12.5% padding
    F32_DMA_CG(181, 2, 7, 4, 4, 16, 3, 3, 3, 11, 1, 5, 4),
    F32_DMA_CG(182, 2, 7, 8, 8, 32, 3, 3, 2, 11, 1, 5, 4),
    F32_DMA_CG(163, 1, 4, 4, 4, 16, 3, 3, 3, 11, 1, 3, 4),
    F32_DMA_CG(164, 2, 4, 8, 4, 16, 3, 3, 2, 8, 1, 5, 4),
    F32_DMA_CG(165, 4, 4, 4, 4, 16, 3, 3, 3, 8, 1, 10, 4),
    F32_DMA_CG(166, 2, 2, 8, 4, 16, 3, 3, 2, 6, 1, 5, 4),
    F32_DMA_CG(167, 4, 2, 8, 4, 16, 3, 3, 2, 8, 1, 5, 4),
    // 2x2 taps (inner problems of stride-2 3x3 layers): deep channel ranges
    F32_DMA_CG(168, 2, 2, 8, 8, 64, 2, 2, 2, 6, 1, 5, 4),
    F32_DMA_CG(169, 2, 2, 4, 4, 32, 2, 2, 3, 6, 1, 5, 4),
    F32_DMA_CG(178, 1, 2, 8, 8, 64, 2, 2, 2, 6, 1, 3, 4),
    // 1x1 taps: deep channel ranges on few pixels
    F32_DMA_CG(171, 2, 2, 4, 4, 64, 1, 1, 3, 9, 1, 3, 4),
    F32_DMA_CG(172, 2, 2, 8, 8, 128, 1, 1, 2, 9, 1, 3, 4),
    F32_DMA_CG(173, 4, 2, 4, 4, 64, 1, 1, 3, 9, 1, 5, 4),
    F32_DMA_CG(174, 4, 4, 4, 4, 64, 1, 1, 3, 17, 1, 5, 4),
    // 32x32x2 inner loop, 3x3 taps: (pixel units of 16 per wave, waves, ...)
    F32_DMA32(151, 4, 4, 8, 3, 3, 3, 12, 1, 10, 4),
    F32_DMA32(152, 4, 4, 8, 3, 3, 3, 7, 1, 19, 1),
    F32_DMA32(153, 4, 8, 8, 3, 3, 3, 4, 1, 10, 1),
    F32_DMA32(154, 2, 8, 8, 3, 3, 3, 5, 1, 19, 1),
    // 1x1 taps
    F32_DMA(131, 4, 7, 4, 16, 1, 1, 3, 7, 4, 5, 1),
    F32_DMA(132, 4, 7, 4, 16, 1, 1, 4, 7, 4, 5, 1),
    F32_DMA(133, 4, 4, 8, 16, 1, 1, 3, 4, 4, 3, 1),
    F32_DMA(134, 4, 8, 4, 16, 1, 1, 3, 8, 4, 5, 1),
    F32_DMA(135, 4, 6, 4, 16, 1, 1, 3, 6, 4, 5, 1),
    F32_DMA(136, 4, 8, 8, 16, 1, 1, 3, 8, 4, 3, 1),
    // scalar In loads: any row length (Q % 4 != 0)
    F32_DMA(137, 4, 4, 4, 16, 1, 1, 3, 17, 1, 5, 4),
    F32_DMA(138, 4, 4, 4, 8, 1, 1, 4, 9, 1, 3, 4),
    F32_DMA(139, 4, 5, 4, 32, 1, 1, 3, 21, 1, 5, 4),
    F32_DMA(140, 4, 4, 4, 32, 1, 1, 3, 17, 1, 5, 4),
    F32_DMA(121, 1, 25, 4, 16, 1, 1, 4, 7, 4, 2, 4),
    F32_DMA(126, 1, 13, 8, 16, 1, 1, 4, 4, 4, 1, 4),
    F32_DMA(127, 1, 7, 8, 16, 1, 1, 4, 2, 4, 1, 4),
    F32_DMA(128, 2, 7, 8, 16, 1, 1, 3, 4, 4, 1, 4),
    F32_DMA(122, 1, 25, 4, 16, 1, 1, 3, 7, 4, 2, 4),
    F32_DMA(123, 4, 4, 4, 16, 1, 1, 3, 4, 4, 2, 4),
    F32_DMA(124, 2, 13, 4, 16, 1, 1, 3, 7, 4, 2, 4),
    F32_DMA(125, 1, 13, 4, 16, 1, 1, 4, 4, 4, 2, 4),
    // ---- bf16 inputs, C = 32: pixel-fastest shifted LDS copies, transposing reads
    // (tile rows, tile columns, taps)
    BF16_TR_INST(211, 7, 64, 3, 3),
    BF16_TR_INST(212, 4, 64, 3, 3),
    BF16_TR_INST(213, 8, 64, 3, 3),
    BF16_TR_INST(214, 8, 32, 3, 3),
    BF16_TR_INST(215, 14, 32, 3, 3),
    BF16_TR_INST(216, 4, 32, 3, 3),
    // ---- bf16 inputs (persistent, transposed channel-fastest LDS tiles)
    BF16_INST(201, 4, 4, 3, 3, 3),
    BF16_INST(202, 2, 4, 3, 3, 3),
    BF16_INST(203, 4, 2, 3, 3, 3),
    BF16_INST(204, 4, 4, 1, 1, 3),
    BF16_INST(205, 2, 2, 3, 3, 3),
    // 2x2 and 4x4 taps: stride-2 3x3 and 7x7 layers after the polyphase rewrite
    BF16_INST(206, 4, 4, 2, 2, 3),
    BF16_INST(207, 4, 4, 4, 4, 3),
    // ---- register-staged, double buffered (any shape, any alignment)
    // 3x3 taps, Ker staged in float4
    F32_INST(1, 4, 4, 8, 3, 3, 8, 12, 4),
    F32_INST(2, 2, 4, 8, 3, 3, 8, 12, 4),
    F32_INST(3, 4, 2, 8, 3, 3, 8, 12, 4),
    F32_INST(4, 2, 2, 8, 3, 3, 8, 12, 4),
    F32_INST(5, 1, 4, 8, 3, 3, 8, 12, 4),
    F32_INST(6, 4, 1, 8, 3, 3, 8, 12, 4),
    F32_INST(7, 2, 2, 4, 3, 3, 8, 12, 4),
    // 1x1 taps
    F32_INST(20, 4, 4, 16, 1, 1, 16, 4, 4),
    F32_INST(21, 2, 4, 16, 1, 1, 16, 4, 4),
    F32_INST(22, 4, 2, 16, 1, 1, 16, 4, 4),
    F32_INST(23, 2, 2, 16, 1, 1, 16, 4, 4),
    F32_INST(24, 4, 4, 8, 1, 1, 8, 4, 4),
    // any taps (runtime R, S), scalar Ker staging: any C, any alignment
    F32_INST(40, 2, 2, 4, 0, 0, 12, 16, 1),
    F32_INST(41, 4, 4, 4, 0, 0, 12, 32, 1),
};

constexpr int kNumInstances = sizeof(kInstances) / sizeof(kInstances[0]);

const Instance* find_instance(int id) {
  for (int i = 0; i < kNumInstances; ++i)
    if (kInstances[i].v.id == id) return &kInstances[i];
  return nullptr;
}

}  // namespace

namespace {
struct VariantTable {
  Variant v[kNumInstances];
  VariantTable() {
    for (int i = 0; i < kNumInstances; ++i) v[i] = kInstances[i].v;
  }
};
}  // namespace

const Variant* variants(int* count) {
  // A function-local static: initialised once, thread-safe (C++11).
  static const VariantTable table;
  *count = kNumInstances;
  return table.v;
}

const Variant* find_variant(int id) {
  const Instance* in = find_instance(id);
  return in ? &in->v : nullptr;
}

// Raise a kernel's dynamic LDS limit to what the CU's 160 KB leave beside
// its static LDS.
int allow_dynamic_lds(const void* fn) {
  hipFuncAttributes attr;
  if (hipFuncGetAttributes(&attr, fn) != hipSuccess) return CONV_EHIP;
  const int limit = 163840 - (int)attr.sharedSizeBytes;
  return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, limit) == hipSuccess ? CONV_OK
                                                                                                  : CONV_EHIP;
}

// Workspaces come from a memory pool the library owns, one per device,
// which keeps up to 1 GB of freed blocks for reuse (the default pool hands
// freed memory back at each synchronisation, so every call would map fresh
// pages).  The calling thread's current device must own the stream.
constexpr int kMaxDevices = 64;

int stream_alloc(size_t bytes, void* stream, void** out) {
  static std::mutex mu;
  static hipMemPool_t pools[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return CONV_EHIP;
  hipMemPool_t pool = nullptr;
  {
    std::lock_guard<std::mutex> lk(mu);
    if (!pools[dev]) {
      hipMemPoolProps props = {};
      props.allocType = hipMemAllocationTypePinned;
      props.location.type = hipMemLocationTypeDevice;
      props.location.id = dev;
      hipMemPool_t p = nullptr;
      if (hipMemPoolCreate(&p, &props) != hipSuccess) return CONV_EHIP;
      uint64_t keep = uint64_t(1) << 30;
      if (hipMemPoolSetAttribute(p, hipMemPoolAttrReleaseThreshold, &keep) != hipSuccess) return CONV_EHIP;
      pools[dev] = p;
    }
    pool = pools[dev];
  }
  return hipMallocFromPoolAsync(out, bytes, pool, reinterpret_cast<hipStream_t>(stream)) == hipSuccess ? CONV_OK
                                                                                                      : CONV_EHIP;
}

int stream_free(void* p, void* stream) {
  return hipFreeAsync(p, reinterpret_cast<hipStream_t>(stream)) == hipSuccess ? CONV_OK : CONV_EHIP;
}

// ---------------------------------------------------------------------------
// Scratch of the allocation-free entry point: a static device array.  Every
// GPU that loads the library's code object holds its own copy (at its own
// address) until the process ends.  Host code must not use the array's name
// as a device address (on the host it names a host-side stand-in); it uses
// the per-device address that hipGetSymbolAddress reports, taken once per
// device with that device current.
static __device__ __align__(256) char scratch[CONV_NOALLOC_SCRATCH_BYTES];

int noalloc_scratch(void** base) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return CONV_EHIP;
  std::lock_guard<std::mutex> lk(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return CONV_EHIP;
    addr[dev] = p;
  }
  *base = addr[dev];
  return CONV_OK;
}

namespace {
// Workspaces kept per (device, stream, nesting level): the kernels of the
// calls on one stream run in stream order, so a call can reuse the buffer
// the previous call on that stream used.  A buffer grows by a stream-ordered
// free and a new allocation; while another host thread holds it, a call
// takes a fresh stream-ordered allocation instead.
struct CachedWorkspace {
  void* ptr = nullptr;
  size_t size = 0;
  bool busy = false;
};
std::mutex g_ws_mu;
std::map<std::tuple<int, void*, int>, CachedWorkspace> g_ws;

// The arena of the calling thread's allocation-free call, if one is running.
thread_local ScratchArena* t_arena = nullptr;
}  // namespace

void set_thread_arena(ScratchArena* a) { t_arena = a; }

int workspace_acquire(int level, size_t bytes, void* stream, Workspace* w) {
  w->cached = false;
  w->arena = false;
  w->level = level;
  if (t_arena) {
    // bump allocation from the caller's scratch, 256-byte aligned
    const size_t off = (t_arena->used + 255) / 256 * 256;
    if (off > t_arena->cap || bytes > t_arena->cap - off) return CONV_ESCRATCH;
    w->ptr = t_arena->base + off;
    w->arena = true;
    t_arena->used = off + bytes;
    return CONV_OK;
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return CONV_EHIP;
  {
    std::lock_guard<std::mutex> lk(g_ws_mu);
    CachedWorkspace& c = g_ws[std::make_tuple(dev, stream, level)];
    if (!c.busy) {
      if (c.size < bytes) {
        if (c.ptr && stream_free(c.ptr, stream) != CONV_OK) return CONV_EHIP;
        c.ptr = nullptr;
        c.size = 0;
        const size_t sz = (bytes + (size_t(1) << 20) - 1) >> 20 << 20;  // whole MiB
        if (stream_alloc(sz, stream, &c.ptr) != CONV_OK) return CONV_EHIP;
        c.size = sz;
      }
      c.busy = true;
      w->ptr = c.ptr;
      w->cached = true;
      return CONV_OK;
    }
  }
  return stream_alloc(bytes, stream, &w->ptr);
}

int workspace_release(const Workspace& w, void* stream) {
  if (w.arena) return CONV_OK;
  if (!w.cached) return stream_free(w.ptr, stream);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return CONV_EHIP;
  std::lock_guard<std::mutex> lk(g_ws_mu);
  g_ws[std::make_tuple(dev, stream, w.level)].busy = false;
  return CONV_OK;
}

int workspace_release_stream(void* stream) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return CONV_EHIP;
  std::lock_guard<std::mutex> lk(g_ws_mu);
  int rc = CONV_OK;
  for (auto it = g_ws.begin(); it != g_ws.end();) {
    if (std::get<0>(it->first) == dev && std::get<1>(it->first) == stream && !it->second.busy) {
      if (it->second.ptr && stream_free(it->second.ptr, stream) != CONV_OK) rc = CONV_EHIP;
      it = g_ws.erase(it);
    } else {
      ++it;
    }
  }
  return rc;
}

int launch_phase_split(const PhaseGeom& p, int dtype, const void* In, const void* Ker, void* Inp, void* Kp,
                       void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int64_t n_in = (int64_t)p.N * p.C * p.na * p.nb * p.Hp * p.Wp;
  const int64_t n_ker = (int64_t)p.K * p.C * p.na * p.nb * p.Rp * p.Sp;
  const int g_in = (int)std::min<int64_t>((n_in + 255) / 256, 8192);
  const int g_ker = (int)std::min<int64_t>((n_ker + 255) / 256, 2048);
  if (dtype == CONV_DTYPE_BF16) {
    if (Inp)
      hipLaunchKernelGGL(phase_split_kernel<unsigned short>, dim3(g_in), dim3(256), 0, st,
                         static_cast<const unsigned short*>(In), static_cast<unsigned short*>(Inp), p);
    if (Kp)
      hipLaunchKernelGGL(ker_phase_kernel<unsigned short>, dim3(g_ker), dim3(256), 0, st,
                         static_cast<const unsigned short*>(Ker), static_cast<unsigned short*>(Kp), p);
  } else {
    if (Inp)
      hipLaunchKernelGGL(phase_split_kernel<float>, dim3(g_in), dim3(256), 0, st, static_cast<const float*>(In),
                         static_cast<float*>(Inp), p);
    if (Kp)
      hipLaunchKernelGGL(ker_phase_kernel<float>, dim3(g_ker), dim3(256), 0, st, static_cast<const float*>(Ker),
                         static_cast<float*>(Kp), p);
  }
  return hipGetLastError() == hipSuccess ? CONV_OK : CONV_EHIP;
}

int launch_widen_bf16(const void* src, float* dst, int64_t n, void* stream) {
  const int blocks = (int)std::max<int64_t>(1, std::min<int64_t>((n + 255) / 256, 8192));
  hipLaunchKernelGGL(widen_bf16_kernel, dim3(blocks), dim3(256), 0, reinterpret_cast<hipStream_t>(stream),
                     static_cast<const unsigned short*>(src), dst, n);
  return hipGetLastError() == hipSuccess ? CONV_OK : CONV_EHIP;
}

int launch_round_bf16(const float* src, void* dst, int64_t n, void* stream) {
  const int blocks = (int)std::max<int64_t>(1, std::min<int64_t>((n + 255) / 256, 8192));
  hipLaunchKernelGGL(round_bf16_kernel, dim3(blocks), dim3(256), 0, reinterpret_cast<hipStream_t>(stream), src,
                     static_cast<unsigned short*>(dst), n);
  return hipGetLastError() == hipSuccess ? CONV_OK : CONV_EHIP;
}

int launch_bf16_out(const Variant& v, const Geom& g, const void* In, const void* Ker, void* Out, void* stream) {
  const Instance* inst = find_instance(v.id);
  if (!inst) return CONV_EINVAL;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (inst->bf16_outb) {
    // lds and alignment as for the fp32-Out launch of the same instance
    static std::mutex mu;
    static bool done[kNumInstances] = {};
    const int idx = (int)(inst - kInstances);
    {
      std::lock_guard<std::mutex> lk(mu);
      if (!done[idx]) {
        if (allow_dynamic_lds(reinterpret_cast<const void*>(inst->bf16_outb)) != CONV_OK) return CONV_EHIP;
        done[idx] = true;
      }
    }
    if ((reinterpret_cast<uintptr_t>(Ker) % 16) != 0) return CONV_EINVAL;
    hipLaunchKernelGGL(inst->bf16_outb, dim3(g.grid), dim3(v.threads), g.stage_elems, st,
                       static_cast<const unsigned short*>(In), static_cast<const unsigned short*>(Ker),
                       static_cast<float*>(Out), g);
    return hipGetLastError() == hipSuccess ? CONV_OK : CONV_EHIP;
  }
  // any other kernel: fp32 Out into a stream-ordered workspace, then rounded
  const int64_t n = (int64_t)g.N * g.K * g.P * g.Q;
  Workspace w;
  int rc = workspace_acquire(1, (size_t)n * sizeof(float), stream, &w);
  if (rc != CONV_OK) return rc;
  void* ws = w.ptr;
  rc = launch(v, g, In, Ker, static_cast<float*>(ws), stream);
  if (rc == CONV_OK) {
    const int blocks = (int)std::min<int64_t>((n + 255) / 256, 8192);
    hipLaunchKernelGGL(round_bf16_kernel, dim3(blocks), dim3(256), 0, st, static_cast<const float*>(ws),
                       static_cast<unsigned short*>(Out), n);
    if (hipGetLastError() != hipSuccess) rc = CONV_EHIP;
  }
  const int freed = workspace_release(w, stream);
  return rc == CONV_OK ? freed : rc;
}

int launch(const Variant& v, const Geom& g, const void* In, const void* Ker, float* Out,
           void* stream) {
  const Instance* inst = find_instance(v.id);
  if (!inst) return CONV_EINVAL;
  int lds_bytes;
  if (v.family == FAMILY_DMA) lds_bytes = v.stages * g.stage_elems * (int)sizeof(float);
  else if (v.family == FAMILY_BF16 || v.family == FAMILY_BF16_TR || v.family == FAMILY_STREAM1X1 ||
           v.family == FAMILY_STREAM1X1_LOOP || v.family == FAMILY_STREAM1X1_BAL)
    lds_bytes = g.stage_elems;  // bytes
  else lds_bytes = 2 * (g.lds_in_elems + g.lds_ker_elems) * (int)sizeof(float);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int ker_elem = v.dtype == CONV_DTYPE_BF16 ? 2 : 4;
  if (v.family != FAMILY_BF16 && v.ker_vec > 1 &&
      (reinterpret_cast<uintptr_t>(Ker) % std::min(16, ker_elem * v.ker_vec)) != 0)
    return CONV_EINVAL;
  const void* fn = inst->f32 ? reinterpret_cast<const void*>(inst->f32)
                             : reinterpret_cast<const void*>(inst->bf16);
  if (g.split > 1 && v.family != FAMILY_DMA) return CONV_EINVAL;
  if (lds_bytes > 65536) {
    // Raise the kernel's dynamic LDS limit once (to the device maximum).
    static std::mutex mu;
    static bool done[kNumInstances] = {};
    const int idx = (int)(inst - kInstances);
    std::lock_guard<std::mutex> lk(mu);
    if (!done[idx]) {
      if (allow_dynamic_lds(fn) != CONV_OK) return CONV_EHIP;
      done[idx] = true;
    }
  }
  if (inst->f32 && g.split > 1) {
    // Split reduction: partial outputs of the channel ranges into a
    // stream-ordered workspace, then the fixed-order sum into Out.
    const int64_t n = (int64_t)g.N * g.K * g.P * g.Q;
    Workspace w;
    const int got = workspace_acquire(2, (size_t)g.split * n * sizeof(float), stream, &w);
    if (got != CONV_OK) return got;
    float* ws = static_cast<float*>(w.ptr);
    hipLaunchKernelGGL(inst->f32, dim3(g.grid), dim3(v.threads), lds_bytes, st,
                       static_cast<const float*>(In), static_cast<const float*>(Ker), ws, g);
    const bool vec4 = (n % 4 == 0) && (reinterpret_cast<uintptr_t>(Out) % 16 == 0);
    const int64_t items = vec4 ? n / 4 : n;
    const int blocks = (int)std::min<int64_t>((items + 255) / 256, 4096);
    if (vec4) hipLaunchKernelGGL(splitk_reduce_kernel<true>, dim3(blocks), dim3(256), 0, st, ws, Out, n, g.split);
    else hipLaunchKernelGGL(splitk_reduce_kernel<false>, dim3(blocks), dim3(256), 0, st, ws, Out, n, g.split);
    const hipError_t launched = hipGetLastError();
    const int freed = workspace_release(w, stream);
    return (launched == hipSuccess && freed == CONV_OK) ? CONV_OK : CONV_EHIP;
  }
  if (inst->f32) {
    hipLaunchKernelGGL(inst->f32, dim3(g.grid), dim3(v.threads), lds_bytes, st,
                       static_cast<const float*>(In), static_cast<const float*>(Ker), Out, g);
  } else {
    hipLaunchKernelGGL(inst->bf16, dim3(g.grid), dim3(v.threads), lds_bytes, st,
                       static_cast<const unsigned short*>(In),
                       static_cast<const unsigned short*>(Ker), Out, g);
  }
  return hipGetLastError() == hipSuccess ? CONV_OK : CONV_EHIP;
}

// Holds the stream for `ticks` of the 100 MHz wall clock (bounded wait), so
// that the launches queued behind it start back to back.
__global__ void delay_kernel(unsigned long long ticks) {
  const unsigned long long t0 = wall_clock64();
  while (wall_clock64() - t0 < ticks) __builtin_amdgcn_s_sleep(8);
}

// Reads n4 float4 of a scratch buffer (its contents are irrelevant), so that
// whatever a timed launch reads afterwards comes from HBM, not from the L2 or
// the last-level cache.  The store never happens in practice; it keeps the
// loads.
__global__ void evict_kernel(const v4f* __restrict__ buf, int64_t n4, float* __restrict__ sink) {
  float acc = 0.f;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n4; i += (int64_t)gridDim.x * blockDim.x) {
    const v4f v = buf[i];
    acc += v[0] + v[1] + v[2] + v[3];
  }
  if (acc == -12345.678f) sink[threadIdx.x] = acc;
}

constexpr size_t kEvictBytes = size_t(512) << 20;  // twice the last-level cache

int time_launches(const Variant& v, const Geom& g, const void* In, const void* Ker, float* Out,
                  void* stream, int reps, float* us) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  int rc = launch(v, g, In, Ker, Out, stream);  // untimed: first-launch set-up, caches
  if (rc != CONV_OK) return rc;
  // Each launch runs after a pass over a 512 MB scratch buffer (so In comes
  // from HBM, as in a network where every call has new data) and between its
  // own two events; all of it queued behind a delay of 300 us per launch, so
  // host time between launches does not count.
  void* evict_buf = nullptr;
  if (stream_alloc(kEvictBytes, stream, &evict_buf) != CONV_OK) return CONV_EHIP;
  std::vector<hipEvent_t> ev(2 * (size_t)reps, nullptr);
  for (auto& e : ev)
    if (rc == CONV_OK && hipEventCreate(&e) != hipSuccess) rc = CONV_EHIP;
  if (rc == CONV_OK) {
    hipLaunchKernelGGL(delay_kernel, dim3(1), dim3(64), 0, st, (unsigned long long)(100ull * 300 * reps));
    if (hipGetLastError() != hipSuccess) rc = CONV_EHIP;
  }
  for (int i = 0; rc == CONV_OK && i < reps; ++i) {
    hipLaunchKernelGGL(evict_kernel, dim3(2048), dim3(256), 0, st, static_cast<const v4f*>(evict_buf),
                       (int64_t)(kEvictBytes / sizeof(v4f)), static_cast<float*>(evict_buf));
    if (hipGetLastError() != hipSuccess) rc = CONV_EHIP;
    if (rc == CONV_OK && hipEventRecord(ev[2 * i], st) != hipSuccess) rc = CONV_EHIP;
    if (rc == CONV_OK) rc = launch(v, g, In, Ker, Out, stream);
    if (rc == CONV_OK && hipEventRecord(ev[2 * i + 1], st) != hipSuccess) rc = CONV_EHIP;
  }
  const bool freed = hipFreeAsync(evict_buf, st) == hipSuccess;
  if (rc == CONV_OK && !freed) rc = CONV_EHIP;
  if (rc == CONV_OK && hipEventSynchronize(ev[2 * reps - 1]) != hipSuccess) rc = CONV_EHIP;
  std::vector<float> t(reps, 0.f);
  for (int i = 0; rc == CONV_OK && i < reps; ++i)
    if (hipEventElapsedTime(&t[i], ev[2 * i], ev[2 * i + 1]) != hipSuccess) rc = CONV_EHIP;
  for (auto& e : ev)
    if (e) (void)hipEventDestroy(e);
  if (rc != CONV_OK) return rc;
  std::sort(t.begin(), t.end());
  *us = t[reps / 2] * 1000.f;  // median
  return CONV_OK;
}

}  // namespace convfwd
