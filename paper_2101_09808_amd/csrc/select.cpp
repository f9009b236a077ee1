// Tile selector for the gfx950 convolution kernels (host only, no HIP calls).
//
// The paper's method (Sec. 3-5, Algorithm 1 of Sec. 8) chooses, for each
// level of the memory hierarchy, a tile-loop permutation from the eight
// pruned classes and tile sizes that minimise the bandwidth-scaled data
// volume of the most constrained level: min over plans of max_l DV^l / BW^l.
// Here the search runs over integer candidates that the kernels can execute
// (tile sizes are multiples of the 16x16 MFMA block; the reduction loops are
// innermost inside a workgroup, i.e. the Out-stationary classes), so the
// max is evaluated directly instead of through region-constrained solves.
//
// Levels (innermost first), and how their volumes follow the paper's model:
//   REG  LDS -> VGPR operand reads.  Inside a wave the accumulator tile is
//        stationary and every operand is read once per (4 channels, tap), so
//        the level behaves like the tiled matmul of Sec. 2.2 over the im2col
//        view: bytes = MACs * (1/T_k + 1/T_px) * 4 (Eq. (3) form, Out moves 0).
//   LDS  L2 -> LDS staging.  Class <{n,k,h,w},{c,r},s> with T_r = R, T_s = S:
//        per workgroup tile, every channel step brings the In halo footprint
//        (T_h + R - 1)(T_w + S - 1) and the Ker footprint T_k*T_c*R*S
//        (Sec. 3.2, first case; Eq. (4) footprints).
//   L2   MALL/HBM -> L2 per XCD: the outer tile-loop order of the grid (k
//        tiles innermost: In stays, Ker re-read unless it fits the XCD's L2;
//        pixel tiles innermost: Ker stays, In re-read per k tile).
//   HBM  compulsory bytes: In + Ker read once, Out written once.
// A compute "level" (MFMA time incl. padding and wave quantisation over the
// 256 CUs) plays the part of the paper's load balancing step.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <map>
#include <mutex>
#include <tuple>
#include <vector>

#include "conv_internal.h"

namespace convfwd {

// ---------------------------------------------------------------------------
// The paper's single-level model, Sec. 3.2.  Iterator codes n=0 k=1 c=2 r=3
// s=4 h=5 w=6.  In is indexed by n, c, h+r, w+s; Ker by k, c, r, s; Out by
// n, k, h, w.
namespace {
enum { IN = 0, KER = 1, OUT = 2 };
const bool kPresent[3][7] = {
    /* In  */ {true, false, true, true, true, true, true},
    /* Ker */ {false, true, true, true, true, false, false},
    /* Out */ {true, true, false, false, false, true, true},
};
}  // namespace

void model_volume(const int perm[7], const int64_t N[7], const int64_t T[7], int out_factor,
                  double dv[3]) {
  // pos[x]: 1 for the innermost loop, 7 for the outermost.
  int pos[7];
  for (int i = 0; i < 7; ++i) pos[perm[i]] = 7 - i;
  const double Tn = (double)T[0], Tk = (double)T[1], Tc = (double)T[2], Tr = (double)T[3],
               Ts = (double)T[4], Th = (double)T[5], Tw = (double)T[6];
  const double foot[3] = {
      Tn * Tc * (Th + Tr - 1) * (Tw + Ts - 1),  // In
      Tk * Tc * Tr * Ts,                        // Ker
      Tn * Tk * Th * Tw,                        // Out
  };
  for (int a = 0; a < 3; ++a) {
    int ra = 8, it = -1;
    for (int x = 0; x < 7; ++x)
      if (kPresent[a][x] && pos[x] < ra) {
        ra = pos[x];
        it = x;
      }
    const bool sliding = (a == IN) && (it == 3 || it == 4 || it == 5 || it == 6);
    double ratio = 1.0;
    for (int x = 0; x < 7; ++x)
      if (sliding ? pos[x] > ra : pos[x] >= ra) ratio *= (double)N[x] / (double)T[x];
    double v;
    if (sliding) {
      // Consecutive tiles along the sliding iterator share all but T_x of
      // their extent in that data dimension: first tile in full, then the
      // extent replaced by N_x - T_x.
      double part;
      if (it == 6) part = Tn * Tc * (Th + Tr - 1) * ((double)N[6] - Tw);
      else if (it == 4) part = Tn * Tc * (Th + Tr - 1) * ((double)N[4] - Ts);
      else if (it == 5) part = Tn * Tc * ((double)N[5] - Th) * (Tw + Ts - 1);
      else part = Tn * Tc * ((double)N[3] - Tr) * (Tw + Ts - 1);
      v = ratio * (foot[IN] + part);
    } else {
      v = ratio * foot[a];
    }
    dv[a] = (a == OUT) ? v * out_factor : v;
  }
}

// ---------------------------------------------------------------------------
// Hardware description of one MI355X (AMD public figures; the LDS and L2
// figures are per-CU port widths times the clock).
namespace {
struct Hw {
  double clock_hz = 2.4e9;
  int cus = 256;
  int xcds = 8;
  int simds_per_cu = 4;
  int lds_bytes = 163840;
  double l2_bytes = 4.0 * 1024 * 1024;  // per XCD
  double bw[CONV_NUM_LVLS] = {
      256 * 128 * 2.4e9,  // REG: LDS read, 128 B/clk/CU
      256 * 64 * 2.4e9,   // LDS: L2 -> CU, 64 B/clk/CU
      17.0e12,            // L2: MALL/fabric -> L2 (aggregate)
      8.0e12,             // HBM
  };
  int mfma_f32_cycles = 32;  // 16x16x4 f32 per SIMD
  double launch_us = 5.0;    // one more kernel launch in the stream: a split plan's reduce pass
                             // measured 4-5 us over the same plan unsplit on small layers
  // Pipeline fill and drain of a launch (Little's law, Sec. 6: the first
  // step's data needs one round trip before any MFMA can start).  Per-wave
  // timestamps of the 3x3 N=1 C=64 layer on MI355X: kernel arguments and
  // index set-up 1.2 us, first loads issued and landed 1.4 us after that;
  // the last stores 0.5 us.
  double fill_us = 2.6;
  double drain_us = 0.5;
};
const Hw kHw;

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Bank-conflict cost of a wave's 64 4-byte LDS reads (addresses in
// elements), for the gfx950 LDS as measured with the bank-conflict counter
// (SQ_LDS_BANK_CONFLICT) on access patterns of known stride and grouping:
// 32 banks of 4 bytes, a wave's ds_read_b32 served 32 lanes at a time
// (lanes 0-31, then 32-63); each half takes as many passes as the most
// distinct addresses that fall into one bank (equal addresses are one
// broadcast).  Returns the sum of passes over the two halves (2 =
// conflict-free).
int conflict_cost(const int* addr) {
  int total = 0;
  for (int grp = 0; grp < 2; ++grp) {
    int worst = 0;
    for (int b = 0; b < 32; ++b) {
      int seen[32], n = 0;
      for (int l = 32 * grp; l < 32 * grp + 32; ++l) {
        if (((addr[l] % 32) + 32) % 32 != b) continue;
        bool dup = false;
        for (int q = 0; q < n; ++q) dup |= seen[q] == addr[l];
        if (!dup) seen[n++] = addr[l];
      }
      worst = std::max(worst, n);
    }
    total += std::max(1, worst);
  }
  return total;
}

// Row pitch of the Ker tile: >= need, a multiple of `mult`, with the least
// conflicted A-operand reads (lane (i, g) reads row i, column g*RS).
int pick_ker_rstride_uncached(int need, int mult, int rs) {
  int best = -1, best_cost = 1 << 30;
  for (int cand = ((need + mult - 1) / mult) * mult; cand < need + 64 + mult; cand += mult) {
    int addr[64];
    for (int l = 0; l < 64; ++l) addr[l] = (l & 15) * cand + (l >> 4) * rs;
    const int c = conflict_cost(addr);
    if (c < best_cost) {
      best_cost = c;
      best = cand;
    }
  }
  return best;
}

// Channel stride of the In tile: >= need, a multiple of 4, least conflicted
// B-operand reads (lane (j, g) reads channel g, pixel j of the tile's first
// 16-pixel block: row j / tw, column j % tw of rows `wp` elements apart).
int pick_in_cstride_uncached(int need, int tw, int wp) {
  int best = -1, best_cost = 1 << 30;
  for (int cand = ((need + 3) / 4) * 4; cand < need + 68; cand += 4) {
    int addr[64];
    for (int l = 0; l < 64; ++l) addr[l] = (l >> 4) * cand + ((l & 15) / tw) * wp + (l & 15) % tw;
    const int c = conflict_cost(addr);
    if (c < best_cost) {
      best_cost = c;
      best = cand;
    }
  }
  return best;
}

// Both searches depend on a few small integers; memoise them.
std::mutex g_pad_mu;
std::map<std::tuple<int, int, int>, int> g_pad_cache;

int pick_ker_rstride(int need, int mult, int rs) {
  const auto key = std::make_tuple(need, mult, rs);
  {
    std::lock_guard<std::mutex> lk(g_pad_mu);
    auto it = g_pad_cache.find(key);
    if (it != g_pad_cache.end()) return it->second;
  }
  const int v = pick_ker_rstride_uncached(need, mult, rs);
  std::lock_guard<std::mutex> lk(g_pad_mu);
  g_pad_cache[key] = v;
  return v;
}

int pick_in_cstride(int need, int tw, int wp) {
  const auto key = std::make_tuple(need, -1 - std::min(tw, 16), wp);
  {
    std::lock_guard<std::mutex> lk(g_pad_mu);
    auto it = g_pad_cache.find(key);
    if (it != g_pad_cache.end()) return it->second;
  }
  const int v = pick_in_cstride_uncached(need, std::min(tw, 16), wp);
  std::lock_guard<std::mutex> lk(g_pad_mu);
  g_pad_cache[key] = v;
  return v;
}

// The problem as the kernels see it: a 1x1 correlation of an H x W plane is
// the same computation on a 1 x (H*W) plane, which lets a workgroup tile span
// whole image rows.
Shape kernel_view(const Shape& s) {
  Shape k = s;
  if (s.R == 1 && s.S == 1) {
    k.W = s.H * s.W;
    k.H = 1;
  }
  return k;
}
}  // namespace

namespace {
FastDiv make_fastdiv(int d) {
  FastDiv f{0u, 0};
  if (d <= 0) return f;
  int s = 0;
  while ((int64_t(1) << s) < d) ++s;
  const uint64_t num = uint64_t(1) << (31 + s);
  f.m = (unsigned)((num + (uint64_t)d - 1) / (uint64_t)d);
  f.s = s;
  return f;
}
}  // namespace

void set_fast_divisors(Geom* g) {
  g->dv_in_cstride = make_fastdiv(g->in_cstride);
  g->dv_in_wp = make_fastdiv(g->in_wp);
  g->dv_H = make_fastdiv(g->H);
  g->dv_ker_rstride = make_fastdiv(g->ker_rstride);
  g->dv_tw = make_fastdiv(g->tw);
  g->dv_P = make_fastdiv(g->P);
  g->dv_nph = make_fastdiv(g->nph);
  g->dv_nb = make_fastdiv(g->nb);
  g->dv_Wi = make_fastdiv(g->Wi);
  g->dv_tiles_k = make_fastdiv(g->tiles_k);
  g->dv_tiles_cols = make_fastdiv(g->tiles_cols);
  g->dv_tiles_rows = make_fastdiv(g->tiles_rows);
}

bool resolve_geom(const Shape& s0, const Variant& v, const conv_plan_t& plan, Geom* g,
                  int* lds_bytes) {
  const Shape s = kernel_view(s0);
  if (plan.dtype != v.dtype) return false;
  const int split = std::max(1, plan.split_c);
  if (split > 1 && v.family != FAMILY_DMA) return false;  // only that kernel splits the reduction
  if (v.family == FAMILY_STREAM1X1 || v.family == FAMILY_STREAM1X1_LOOP) {
    // Pointwise streaming: tile_cols = pixels per wave, 4 waves per workgroup,
    // 64 output channels per workgroup, the whole channel range resident.
    if (s0.R != 1 || s0.S != 1) return false;
    if (plan.tile_k != 64 || plan.waves_k != 1 || plan.waves_px != 4 || plan.tile_rows != 1) return false;
    if (plan.wave_k != 64 || plan.wave_px != 16 * v.wp || plan.tile_c != v.tc) return false;
    if (s.C % 4) return false;  // whole channel quads
    const bool unrolled = v.family == FAMILY_STREAM1X1;
    if (unrolled && v.tc != s.C) return false;  // compiled for this channel count
    const int wpx = plan.tile_cols;
    if (wpx < 1 || wpx > 16 * v.wp) return false;
    const int64_t total_px = (int64_t)s.N * s.W;
    const int64_t groups = cdiv(total_px, 4 * (int64_t)wpx);
    const int64_t tiles_k = cdiv(s.K, 64);
    // stored channels: exactly C (unrolled), or C padded to whole loop trips
    const int64_t cst = unrolled ? s.C : cdiv(s.C / 4, v.stages) * v.stages * 4;
    const int64_t bytes = (cst + 1) * 64 * 4;  // Ker rows [k][c] + 1 pad
    if (bytes > kHw.lds_bytes || groups * tiles_k >= (int64_t(1) << 31)) return false;
    if ((int64_t)s.N * s.C * s.W * 4 >= (int64_t(1) << 30)) return false;  // 32-bit byte offsets
    if ((int64_t)s.K * s.C * 4 >= (int64_t(1) << 31)) return false;        // below the Ker sentinel
    Geom q;
    std::memset(&q, 0, sizeof(q));
    q.N = s.N; q.C = s.C; q.K = s.K; q.H = s.H; q.W = s.W; q.R = 1; q.S = 1;
    q.P = s.P(); q.Q = s.Q();
    q.tr = 1; q.tw = wpx;
    q.tiles_rows = (int)groups; q.tiles_cols = 1; q.tiles_k = (int)tiles_k;
    q.nwk = 1; q.nwp = 4;
    q.num_tiles = (int)(groups * tiles_k);
    q.grid = q.num_tiles;
    q.nchunks = (int)cdiv(s.C, 4);
    q.split = 1;
    q.cps = q.nchunks;
    q.stage_elems = (int)bytes;
    q.in_bytes = (unsigned)std::min<int64_t>((int64_t)s.N * s.C * s.H * s.W * 4, 0xffffffffLL);
    q.ker_bytes = (unsigned)std::min<int64_t>((int64_t)s.K * s.C * 4, 0xffffffffLL);
    if (g) {
      set_fast_divisors(&q);
      *g = q;
    }
    if (lds_bytes) *lds_bytes = (int)bytes;
    return true;
  }
  if (v.family == FAMILY_STREAM1X1_BAL) {
    // Balanced pointwise: tile_cols = pixels per workgroup PW, with
    // 128 NB < PW <= 128 NB + 16 (NB 32-pixel blocks per wave, the rest one
    // 16-pixel block split by k, which counts as one more 16-pixel unit of
    // each wave: wave_px = 32 NB + 16); 64 output channels per workgroup, the
    // whole channel range resident.
    if (s0.R != 1 || s0.S != 1) return false;
    if (plan.tile_k != 64 || plan.waves_k != 1 || plan.waves_px != 4 || plan.tile_rows != 1) return false;
    if (plan.wave_k != 64 || plan.wave_px != 16 * v.wp || plan.tile_c != v.tc || v.tc != s.C) return false;
    if (s.C % 64) return false;
    const int pw = plan.tile_cols, nb = v.max_ni;
    if (pw <= 128 * nb || pw > 128 * nb + 16) return false;
    const int64_t total_px = (int64_t)s.N * s.W;
    const int64_t groups = cdiv(total_px, pw);
    const int64_t tiles_k = cdiv(s.K, 64);
    const int64_t bytes = (int64_t)(s.C + 1) * 64 * 4;  // Ker rows [k][c] + 1 pad
    if (bytes > kHw.lds_bytes || groups * tiles_k >= (int64_t(1) << 31)) return false;
    if ((int64_t)s.N * s.C * s.W * 4 >= (int64_t(1) << 30)) return false;  // 32-bit byte offsets
    if ((int64_t)s.K * s.C * 4 >= (int64_t(1) << 31)) return false;        // below the Ker sentinel
    if ((int64_t)s.N * s.K * s.W * 4 >= (int64_t(1) << 31)) return false;  // Out: 32-bit store offsets
    Geom q;
    std::memset(&q, 0, sizeof(q));
    q.N = s.N; q.C = s.C; q.K = s.K; q.H = s.H; q.W = s.W; q.R = 1; q.S = 1;
    q.P = s.P(); q.Q = s.Q();
    q.tr = 1; q.tw = pw;
    q.tiles_rows = (int)groups; q.tiles_cols = 1; q.tiles_k = (int)tiles_k;
    q.nwk = 1; q.nwp = 4;
    q.num_tiles = (int)(groups * tiles_k);
    q.grid = q.num_tiles;
    q.nchunks = (int)cdiv(s.C, 4);
    q.split = 1;
    q.cps = q.nchunks;
    q.stage_elems = (int)bytes;
    q.in_bytes = (unsigned)std::min<int64_t>((int64_t)s.N * s.C * s.H * s.W * 4, 0xffffffffLL);
    q.ker_bytes = (unsigned)std::min<int64_t>((int64_t)s.K * s.C * 4, 0xffffffffLL);
    if (g) {
      set_fast_divisors(&q);
      *g = q;
    }
    if (lds_bytes) *lds_bytes = (int)bytes;
    return true;
  }
  if (v.rc && (s.R != v.rc || s.S != v.sc)) return false;
  if (plan.tile_c != v.tc) return false;
  const int nwk = plan.waves_k, nwp = plan.waves_px;
  if (nwk < 1 || nwp < 1 || nwk * nwp * v.groups() * 64 != v.threads) return false;
  const int BK = 16 * v.wk * nwk, BP = 16 * v.wp * nwp;
  if (plan.tile_k != BK || plan.wave_k != 16 * v.wk || plan.wave_px != 16 * v.wp) return false;
  if (plan.grid_order != 0 && plan.grid_order != 1) return false;
  const int P = s.P(), Q = s.Q();
  const int tr = plan.tile_rows, tw = plan.tile_cols;
  if (tw < 1 || tw > Q || tr < 1 || (int64_t)tr * tw > BP) return false;
  const int64_t NP = (int64_t)s.N * P;
  const int64_t tiles_rows = cdiv(NP, tr), tiles_cols = cdiv(Q, tw), tiles_k = cdiv(s.K, BK);
  const int64_t num_tiles = tiles_rows * tiles_cols * tiles_k;
  if (num_tiles <= 0 || num_tiles >= (int64_t(1) << 31)) return false;
  // Input rows (flattened n*H + y) spanned by the worst row tile.
  int in_rows = 0;
  for (int64_t rt = 0; rt < tiles_rows; ++rt) {
    const int64_t r0 = rt * tr, r1 = std::min<int64_t>(r0 + tr, NP) - 1;
    const int64_t nu0 = (r0 / P) * s.H + r0 % P, nu1 = (r1 / P) * s.H + r1 % P + s.R - 1;
    in_rows = std::max<int>(in_rows, (int)(nu1 - nu0 + 1));
  }
  const int RS = s.R * s.S, TC = v.tc;
  if (v.family == FAMILY_BF16_TR) {
    // C = 32 and K <= 64 (one channel chunk, one k tile), W even (dword
    // loads of pixel pairs) and at least 8 (a row's last 8 pixels are one
    // 16-byte load), columns in blocks of 16, every block of the tile owned
    // by a wave.  In and Out below 2 GB (32-bit buffer offsets).  LDS: Ker [64][taps][64 B] + S shifted copies of
    // the In tile [32 c][in_rows][tw] bf16, channel planes padded to
    // 16 (mod 64) elements so a transposing read's four channels hit
    // distinct banks.
    // Compile-time tile: max_ni rows x max_nk columns, P a multiple of the
    // rows (a tile never straddles two images).
    if (s.C != 32 || s.K > 64 || s.W % 2 || s.W < 8 || nwk != 1 || plan.grid_order != 1) return false;
    if (tr != v.max_ni || tw != v.max_nk || P % tr) return false;
    const int kpitch = (RS & 1) ? RS : RS + 1;
    int64_t cp = (int64_t)in_rows * tw;
    cp += (16 - cp % 64 + 64) % 64;
    const int64_t bytes_t = (int64_t)64 * kpitch * 64 + (int64_t)s.S * 32 * cp * 2;
    if (bytes_t > kHw.lds_bytes || in_rows != tr + s.R - 1) return false;
    if ((int64_t)s.N * 32 * s.H * s.W * 2 >= (int64_t(1) << 31)) return false;  // below the sentinel
    if ((int64_t)s.N * s.K * P * Q * 4 >= (int64_t(1) << 31)) return false;
    Geom q;
    std::memset(&q, 0, sizeof(q));
    q.N = s.N; q.C = s.C; q.K = s.K; q.H = s.H; q.W = s.W; q.R = s.R; q.S = s.S;
    q.P = P; q.Q = Q;
    q.tr = tr; q.tw = tw;
    q.tiles_rows = (int)tiles_rows; q.tiles_cols = (int)tiles_cols; q.tiles_k = (int)tiles_k;
    q.in_rows = in_rows; q.in_wp = tw; q.in_cstride = (int)cp;
    q.ker_rstride = kpitch;
    q.nwk = nwk; q.nwp = nwp;
    q.order = 1;
    q.num_tiles = (int)num_tiles;
    q.nchunks = 1;
    q.split = 1;
    q.cps = 1;
    q.stage_elems = (int)bytes_t;
    q.grid = (int)std::min<int64_t>(num_tiles, (int64_t)kHw.cus);
    q.in_bytes = (unsigned)((int64_t)s.N * s.C * s.H * s.W * 2);
    q.ker_bytes = (unsigned)std::min<int64_t>((int64_t)s.K * s.C * RS * 2, 0xffffffffLL);
    if (g) {
      set_fast_divisors(&q);
      *g = q;
    }
    if (lds_bytes) *lds_bytes = (int)bytes_t;
    return true;
  }
  if (v.family == FAMILY_BF16) {
    // LDS: Ker [BK][RS or RS+1 taps][64 B] + In [in_rows][in_wp][64 B] (bytes)
    const int in_wp_b = ((tw + s.S - 1) + 1) & ~1;
    const int kpitch = (RS & 1) ? RS : RS + 1;
    const int64_t bytes_b = (int64_t)BK * kpitch * 64 + (int64_t)in_rows * in_wp_b * 64;
    if (bytes_b > kHw.lds_bytes) return false;
    if ((int64_t)4 * in_rows * (in_wp_b / 2) > (int64_t)v.max_ni * v.threads) return false;
    Geom q;
    std::memset(&q, 0, sizeof(q));
    q.N = s.N; q.C = s.C; q.K = s.K; q.H = s.H; q.W = s.W; q.R = s.R; q.S = s.S;
    q.P = P; q.Q = Q;
    q.tr = tr; q.tw = tw;
    q.tiles_rows = (int)tiles_rows; q.tiles_cols = (int)tiles_cols; q.tiles_k = (int)tiles_k;
    q.in_rows = in_rows; q.in_wp = in_wp_b; q.in_cstride = 0;
    q.ker_rstride = kpitch;
    q.nwk = nwk; q.nwp = nwp;
    q.order = plan.grid_order;
    q.num_tiles = (int)num_tiles;
    q.nchunks = (int)cdiv(s.C, TC);
    q.split = 1;
    q.cps = q.nchunks;
    q.stage_elems = (int)bytes_b;
    const int occ = std::max(1, std::min(2, (int)(kHw.lds_bytes / bytes_b)));
    q.grid = (int)std::min<int64_t>(num_tiles, (int64_t)kHw.cus * occ);
    q.in_bytes = (unsigned)std::min<int64_t>((int64_t)s.N * s.C * s.H * s.W * 2, 0xffffffffLL);
    q.ker_bytes = (unsigned)std::min<int64_t>((int64_t)s.K * s.C * RS * 2, 0xffffffffLL);
    if (g) {
      set_fast_divisors(&q);
      *g = q;
    }
    if (lds_bytes) *lds_bytes = (int)bytes_b;
    return true;
  }
  const int in_wp = tw + s.S - 1;
  const int64_t E = (int64_t)in_rows * in_wp;
  if (E * TC >= (1 << 20)) return false;
  const int in_cstride = pick_in_cstride((int)E, tw, in_wp);
  const int TCRS = TC * RS;
  if (v.ker_vec > 1 && ((int64_t)s.C * RS % v.ker_vec != 0 || TCRS % v.ker_vec != 0)) return false;
  if (TCRS >= (1 << 16) || BK >= (1 << 15)) return false;
  const int ker_rstride = pick_ker_rstride(TCRS, std::max(4, v.ker_vec), RS);
  const int64_t in_elems_total = (int64_t)s.N * s.C * s.H * s.W;
  const int64_t ker_elems_total = (int64_t)s.K * s.C * RS;
  int64_t lds_in, lds_ker, bytes, ni_in, ni_ker, stage = 0, in_region = 0;
  if (v.family == FAMILY_DMA) {
    // Byte offsets of the buffer loads are 32-bit with an out-of-range
    // marker at 2^31: both tensors must stay below 2 GB.
    if (in_elems_total * 4 >= (int64_t(1) << 31) || ker_elems_total * 4 >= (int64_t(1) << 31))
      return false;
    if (v.in_vec == 4) {
      // Vector In loads need whole, aligned 4-element groups that never
      // straddle a row or the tile edge: pointwise taps, rows and tiles in
      // multiples of 4 elements.
      if (s.R != 1 || s.S != 1 || s.W % 4 || tw % 4 || Q % 4) return false;
    } else if (v.in_vec != 1) {
      return false;
    }
    const int64_t nw = v.threads / 64;
    in_region = (int64_t)v.max_ni * nw * 64 * v.in_vec;
    const int64_t ker_region = (int64_t)v.max_nk * nw * 64 * v.ker_vec;
    lds_in = (int64_t)TC * in_cstride;
    lds_ker = (int64_t)BK * ker_rstride;
    if (in_cstride % v.in_vec || lds_in > in_region || lds_ker > ker_region) return false;
    stage = in_region + ker_region;
    bytes = (int64_t)v.stages * stage * 4;
    ni_in = v.max_ni;
    ni_ker = v.max_nk;
  } else {
    lds_in = (int64_t)TC * in_cstride;
    lds_ker = ((int64_t)BK * ker_rstride + 3) / 4 * 4;
    bytes = 2 * (lds_in + lds_ker) * 4;
    ni_in = cdiv(TC * E, v.threads);
    ni_ker = cdiv((int64_t)BK * TCRS / v.ker_vec, v.threads);
    if (ni_in > v.max_ni || ni_ker > v.max_nk) return false;
  }
  if (bytes > kHw.lds_bytes) return false;
  Geom q;
  std::memset(&q, 0, sizeof(q));
  q.N = s.N; q.C = s.C; q.K = s.K; q.H = s.H; q.W = s.W; q.R = s.R; q.S = s.S;
  q.P = P; q.Q = Q;
  q.tr = tr; q.tw = tw;
  q.tiles_rows = (int)tiles_rows; q.tiles_cols = (int)tiles_cols; q.tiles_k = (int)tiles_k;
  q.in_rows = in_rows; q.in_wp = in_wp; q.in_cstride = in_cstride;
  q.ker_rstride = ker_rstride;
  q.nwk = nwk; q.nwp = nwp;
  q.order = plan.grid_order;
  q.num_tiles = (int)num_tiles;
  q.lds_in_elems = (int)lds_in; q.lds_ker_elems = (int)lds_ker;
  q.ni_in = (int)ni_in; q.ni_ker = (int)ni_ker;
  q.nchunks = (int)cdiv(s.C, TC);
  // Channel ranges: split ranges of cps pipeline steps each, none empty; the
  // workgroups of range r follow those of range r-1.
  q.split = split;
  q.cps = (int)cdiv(q.nchunks, split);
  if ((int64_t)(split - 1) * q.cps >= q.nchunks) return false;
  if (num_tiles * split >= (int64_t(1) << 31)) return false;
  if (split > 1 && (int64_t)split * s.N * s.K * P * Q >= (int64_t(1) << 31)) return false;  // workspace
  q.in_bytes = (unsigned)std::min<int64_t>(in_elems_total * 4, 0xffffffffLL);
  q.ker_bytes = (unsigned)std::min<int64_t>(ker_elems_total * 4, 0xffffffffLL);
  q.stage_elems = (int)stage;
  q.in_region = (int)in_region;
  q.grid = (int)(num_tiles * split);
  if (g) {
    set_fast_divisors(&q);
    *g = q;
  }
  if (lds_bytes) *lds_bytes = (int)bytes;
  return true;
}

namespace {
// Ranking time of a scored plan: predicted time times the kernel variant's
// measured factor.
double rank_time(const conv_plan_t& p) { return p.rank_us; }
}  // namespace

bool phase_direct(const Variant& v, const PhaseGeom& p, int dtype, Geom* g) {
  const int nph = p.na * p.nb;
  if (dtype != CONV_DTYPE_F32) return false;
  const int64_t in_bytes = (int64_t)p.N * p.C * p.H * p.W * 4;
  if (v.family == FAMILY_STREAM1X1_BAL) {
    // a 1x1 layer has one phase; each lane's In offset is mapped once, and
    // the kernel's channel steps keep its offsets below 2^32 for In < 1 GB
    if (nph != 1 || p.Rp != 1 || p.Sp != 1 || in_bytes >= (int64_t(1) << 30)) return false;
  } else {
    if (v.family != FAMILY_DMA || v.in_vec != 1 || v.tc % nph) return false;
    if (in_bytes >= (int64_t(1) << 31)) return false;  // 32-bit byte offsets below the out-of-range marker
  }
  // phase skip: stride 2 along both axes with odd taps (four phases whose
  // zero taps are the last row / column of the odd phases)
  if (v.phase_skip && !(p.na == 2 && p.nb == 2 && p.sh == 2 && p.sw == 2 && p.R == 2 * p.Rp - 1 &&
                        p.S == 2 * p.Sp - 1 && v.tc % 16 == 0))
    return false;
  g->nph = nph;
  g->na = p.na; g->nb = p.nb;
  g->sh = p.sh; g->sw = p.sw;
  g->ph = p.ph; g->pw = p.pw;
  g->C0 = p.C; g->H0 = p.H; g->W0 = p.W;
  g->Wi = (p.Rp == 1 && p.Sp == 1) ? p.Wp : 0;  // kernel_view flattens 1x1 problems
  g->in_bytes = (unsigned)in_bytes;
  set_fast_divisors(g);
  return true;
}

namespace {
double calibration(const Variant& v);

// Paper's Sec. 3.2 volumes (In, Ker, Out elements) of the class
// <{n,k,h,w},{c,r},s> representative n,k,h,w,c,r,s for extents Ne and tile T
// (codes n=0 k=1 c=2 r=3 s=4 h=5 w=6).
void class3_volume(const int64_t Ne[7], const int64_t T[7], int out_factor, double dv[3]) {
  static const int perm[7] = {0, 1, 5, 6, 2, 3, 4};
  model_volume(perm, Ne, T, out_factor, dv);
}

int score_plan_impl(const Shape& s0, conv_plan_t* plan);
}  // namespace

// Fill the model fields of a plan whose tile fields are set.  0 or an error.
int score_plan(const Shape& s0, conv_plan_t* plan) {
  conv_plan_t p = *plan;
  for (int l = 0; l < CONV_NUM_LVLS; ++l) {
    p.class_lvl[l] = 0;
    p.pred_bytes[l] = p.pred_us[l] = p.paper_bytes[l] = 0.0;
  }
  p.pred_mfma_us = p.pred_total_us = p.rank_us = 0.0;
  const int st = score_plan_impl(s0, &p);
  if (st != CONV_OK) return st;
  // HBM: compulsory In + Ker + Out, the full-tile case of Sec. 3.2 (Out
  // written once: the accumulators never leave the registers mid-reduction)
  const Shape s = s0;
  const double e = (p.dtype == CONV_DTYPE_BF16) ? 2.0 : 4.0;
  const int64_t Ne[7] = {s.N, s.K, s.C, s.R, s.S, s.P(), s.Q()};
  double dv[3];
  class3_volume(Ne, Ne, 1, dv);
  p.paper_bytes[CONV_LVL_HBM] = (dv[0] + dv[1]) * e + dv[2] * 4.0;
  p.rank_us = p.pred_total_us * calibration(*find_variant(p.variant));
  *plan = p;
  return CONV_OK;
}

namespace {
int score_plan_impl(const Shape& s0, conv_plan_t* plan) {
  const Variant* v = find_variant(plan->variant);
  if (!v) return CONV_EINVAL;
  Geom g;
  int lds = 0;
  if (!resolve_geom(s0, *v, *plan, &g, &lds)) return CONV_EINVAL;
  const Shape s = kernel_view(s0);
  const double e = (plan->dtype == CONV_DTYPE_BF16) ? 2.0 : 4.0;
  if (v->family == FAMILY_STREAM1X1 || v->family == FAMILY_STREAM1X1_LOOP) {
    // In moves HBM -> VGPR once; Ker slices are staged into LDS once per
    // workgroup; A operands are 4 B LDS reads.
    plan->lds_bytes = lds;
    plan->num_wg = g.grid;
    const double in_b = (double)s.N * s.C * s.W * 4.0, ker_b = (double)s.K * s.C * 4.0;
    const double out_b = (double)s.N * s.K * s.W * 4.0;
    const double waves = (double)g.grid * 4;
    const double nq = std::ceil(s.C / 4.0);
    // A operands per lane and channel quad: 16 B per pass over the channels
    // (the looped kernel makes one pass per phase); each wave of the unrolled
    // kernel reads 16 B for its 32-pixel blocks and 16 B for a 16-pixel block
    auto unit_reads = [](int u) { return (u >= 2 ? 16.0 : 0.0) + (u % 2 ? 16.0 : 0.0); };
    const double a_bytes = v->family == FAMILY_STREAM1X1 ? unit_reads(v->max_ni) + unit_reads(v->max_nk)
                                                         : 16.0 * (v->max_nk > 0 ? 2 : 1);
    plan->pred_bytes[CONV_LVL_REG] = waves * nq * 64 * a_bytes;
    plan->pred_bytes[CONV_LVL_LDS] = (double)g.grid * s.C * 64 * 4.0;
    plan->pred_bytes[CONV_LVL_L2] = in_b * g.tiles_k + ker_b * std::min<double>(g.tiles_rows, kHw.xcds);
    plan->pred_bytes[CONV_LVL_HBM] = in_b + ker_b + out_b;
    plan->class_lvl[CONV_LVL_REG] = 3;
    plan->class_lvl[CONV_LVL_LDS] = 3;
    plan->class_lvl[CONV_LVL_L2] = 1;
    plan->class_lvl[CONV_LVL_HBM] = 0;
    double tmax = 0;
    for (int l = 0; l < CONV_NUM_LVLS; ++l) {
      plan->pred_us[l] = plan->pred_bytes[l] / kHw.bw[l] * 1e6;
      tmax = std::max(tmax, plan->pred_us[l]);
    }
    const double nb = v->wp;
    const double rounds = std::ceil((double)g.grid / kHw.cus);
    // MFMA issue efficiency of the channel loop, measured with per-wave
    // timestamps on the 1x1 N=32 C=256 K=64 layer: 88% with one wave per
    // SIMD; a second wave per SIMD (unrolled kernel with max_nk > 0) hides
    // the operand waits and measured 9% faster
    const bool two_waves = v->family == FAMILY_STREAM1X1 && v->max_nk > 0;
    double issue_eff = two_waves ? 0.96 : 0.88;
    // A pixel range that is not a whole number of 16-pixel blocks masks part
    // of its last block and starts the next wave's range off a 64-byte
    // boundary: measured 17-28% slower than whole blocks at the same MFMA
    // count (60 plans of the 1x1 N=32 C=256 K=64 layer).
    if (g.tw % 16) issue_eff *= 0.8;
    plan->pred_mfma_us = rounds * nb * 4 * nq * kHw.mfma_f32_cycles / kHw.clock_hz * 1e6 / issue_eff;
    // fill: the first Ker chunk and ring; drain: the last block's stores
    plan->pred_total_us = std::max(tmax, plan->pred_mfma_us) + kHw.fill_us + kHw.drain_us;
    return CONV_OK;
  }
  if (v->family == FAMILY_STREAM1X1_BAL) {
    // In moves HBM -> VGPR once; the Ker slice is staged into LDS once per
    // workgroup; per channel quad each wave reads 16 B of A operands per
    // lane for its 32-pixel block and 4 B for its quarter of the tail block.
    plan->lds_bytes = lds;
    plan->num_wg = g.grid;
    const double in_b = (double)s.N * s.C * s.W * 4.0, ker_b = (double)s.K * s.C * 4.0;
    const double out_b = (double)s.N * s.K * s.W * 4.0;
    const double waves = (double)g.grid * 4;
    const double nq = s.C / 4.0, nb = v->max_ni;
    plan->pred_bytes[CONV_LVL_REG] = waves * nq * 64 * (16.0 * nb + 4.0);
    plan->pred_bytes[CONV_LVL_LDS] = (double)g.grid * s.C * 64 * 4.0;
    plan->pred_bytes[CONV_LVL_L2] = in_b * g.tiles_k + ker_b * std::min<double>(g.tiles_rows, kHw.xcds);
    plan->pred_bytes[CONV_LVL_HBM] = in_b + ker_b + out_b;
    plan->class_lvl[CONV_LVL_REG] = 3;
    plan->class_lvl[CONV_LVL_LDS] = 3;
    plan->class_lvl[CONV_LVL_L2] = 1;
    plan->class_lvl[CONV_LVL_HBM] = 0;
    double tmax = 0;
    for (int l = 0; l < CONV_NUM_LVLS; ++l) {
      plan->pred_us[l] = plan->pred_bytes[l] / kHw.bw[l] * 1e6;
      tmax = std::max(tmax, plan->pred_us[l]);
    }
    // per wave and channel quad: 4 32x32x2 MFMAs (twice the 16x16x4 time)
    // per block and one 16x16x4 for the tail; one wave per SIMD
    const double rounds = std::ceil((double)g.grid / kHw.cus);
    const double cycles = nq * (nb * 4 * 2 * kHw.mfma_f32_cycles + kHw.mfma_f32_cycles);
    plan->pred_mfma_us = rounds * cycles / kHw.clock_hz * 1e6 / 0.92;
    plan->pred_total_us = std::max(tmax, plan->pred_mfma_us) + kHw.fill_us + kHw.drain_us;
    return CONV_OK;
  }
  const int RS = s.R * s.S;
  const int64_t NP = (int64_t)s.N * g.P;
  plan->lds_bytes = lds;
  plan->num_wg = g.grid;
  plan->split_c = g.split;

  // REG: per wave and per (4 channels, tap), WK + WP operand reads of 64
  // lanes; the 32x32x2 loop reads 2 + WP/2 operands per (2 channels, tap).
  // (Channel groups of waves share each tile's steps: the count per tile is
  // the same.)
  const int kdepth = (plan->dtype == CONV_DTYPE_BF16) ? 32 : 4;  // reduction per MFMA
  const double steps = (double)g.nchunks * (v->tc / kdepth) * RS;
  // REG: Eq. (3)'s form over the im2col view -- the tiled matmul of Sec. 2.2
  // with the reduction (c, r, s) innermost inside the wave tile, i.e. the
  // class <{n,k,h,w},{c,r},s> volume with n = r = s = h = 1, c = the
  // C*R*S reduction and w = the pixels: operand elements read from LDS =
  // MACs * (1/T_k + 1/T_px).  Extents are rounded up to whole workgroup
  // tiles (partial tiles are computed in full).
  {
    const int64_t kpad = (int64_t)g.tiles_k * g.nwk * 16 * v->wk;
    const int64_t pxpad = (int64_t)g.tiles_rows * g.tiles_cols * g.nwp * 16 * v->wp;
    const int64_t cpad = (int64_t)g.nchunks * v->tc * RS;
    const int64_t Nr[7] = {1, kpad, cpad, 1, 1, 1, pxpad};
    const int64_t Tr[7] = {1, 16 * v->wk, v->mfma32 ? 2 : kdepth, 1, 1, 1, 16 * v->wp};
    double dv[3];
    class3_volume(Nr, Tr, 0, dv);
    plan->pred_bytes[CONV_LVL_REG] = (dv[0] + dv[1]) * e;
    if (v->phase_skip)  // the operands of the zero-tap steps are not read
      plan->pred_bytes[CONV_LVL_REG] *= (2.0 * v->rc - 1) * (2.0 * v->sc - 1) / (4.0 * v->rc * v->sc);
    plan->paper_bytes[CONV_LVL_REG] = plan->pred_bytes[CONV_LVL_REG];
  }

  // LDS: per workgroup, every channel brings its In halo rows and Ker rows.
  // Memory moves whole 128-byte lines (Sec. 12 names spatial locality as the
  // model's missing refinement): a contiguous run of L bytes at a random
  // element alignment touches on average (L + 128 - e) / 128 lines, so each
  // run is charged L + 128 - e bytes.  A tile's rows are runs of their own,
  // unless the rows are so short that their lines overlap: a tile never
  // touches more than the lines of the span from its first to its last
  // element.  A Ker tile holding every channel is one run per k.
  const double line = 128.0;
  auto run_bytes = [&](double L) { return L > 0 ? L + line - e : 0.0; };
  double in_tiles = 0;  // sum over pixel tiles of the halo footprint, bytes per channel, in lines
  std::vector<double> tile_halo((size_t)g.tiles_rows * g.tiles_cols);  // the same per tile rt * tiles_cols + ct
  for (int64_t rt = 0; rt < g.tiles_rows; ++rt) {
    const int64_t r0 = rt * g.tr, r1 = std::min<int64_t>(r0 + g.tr, NP) - 1;
    const int64_t nu0 = (r0 / g.P) * s.H + r0 % g.P, nu1 = (r1 / g.P) * s.H + r1 % g.P + s.R - 1;
    const double rows = (double)(nu1 - nu0 + 1);
    for (int64_t ct = 0; ct < g.tiles_cols; ++ct) {
      const int64_t cols = std::min<int64_t>(g.tw, g.Q - ct * g.tw) + s.S - 1;
      const double span = run_bytes(((rows - 1) * s.W + cols) * e);
      const double t = std::min(span, rows * run_bytes((double)cols * e));
      tile_halo[(size_t)(rt * g.tiles_cols + ct)] = t * s.C;
      in_tiles += t;
    }
  }
  const double in_halo_bytes = in_tiles * s.C;          // one pass over all pixel tiles
  const double ker_bytes = (double)s.K * s.C * RS * e;  // whole kernel tensor (compulsory)
  const double ker_line_bytes =                         // the same, fetched in tiles of lines
      v->tc >= s.C ? (double)s.K * run_bytes((double)s.C * RS * e)
                   : (double)s.K * g.nchunks * run_bytes((double)v->tc * RS * e);
  const double pix_tiles = (double)g.tiles_rows * g.tiles_cols;
  plan->pred_bytes[CONV_LVL_LDS] = in_halo_bytes * g.tiles_k + ker_line_bytes * pix_tiles;
  // The same level before line rounding: the Sec. 3.2 volume of class
  // <{n,k,h,w},{c,r},s> for the workgroup tile (T_k = tile_k, T_c = channels
  // per step, T_r = R, T_s = S; tile_rows rows of one image, or whole images
  // when the tile spans several; T_w = tile_cols), Out kept in registers.
  // Extents are rounded up to whole tiles (partial tiles staged in full).
  // Exact for tiles that divide the layer; a row tile that straddles two
  // images stages R - 1 more rows than this counts.
  {
    const int tr = g.tr, P = g.P;
    const int64_t Tn = tr > P ? tr / P : 1, Th = tr > P ? P : tr;
    const int64_t Tt[7] = {Tn, (int64_t)g.nwk * 16 * v->wk, v->tc, s.R, s.S, Th, g.tw};
    const int64_t Nt[7] = {(s.N + Tn - 1) / Tn * Tn, (int64_t)g.tiles_k * Tt[1], (int64_t)g.nchunks * v->tc, s.R, s.S,
                           (P + Th - 1) / Th * Th, (int64_t)g.tiles_cols * g.tw};
    double dv[3];
    class3_volume(Nt, Tt, 0, dv);
    plan->paper_bytes[CONV_LVL_LDS] = (dv[0] + dv[1]) * e;
  }

  // L2: outer tile-loop order of the grid, per XCD.
  const double in_bytes = (double)s.N * s.C * s.H * s.W * e;
  const double out_bytes = (double)s.N * s.K * g.P * g.Q * 4.0;
  const bool one_tile_per_wg = v->family == FAMILY_DMA || v->family == FAMILY_STAGED;
  if (one_tile_per_wg && g.split == 1 && g.grid == g.num_tiles && g.grid <= kHw.cus) {
    // One round: every tile is in flight at once.  Workgroup b runs on XCD
    // b mod 8 and takes tile L = xcd_remap(b), so each XCD holds one
    // contiguous range of L (and at most one of the last G mod 8 tiles); its
    // L2 fetches each In halo tile and each k slice of Ker that the range
    // touches once.  With k tiles innermost (order 0) a range spans few
    // pixel tiles and every k slice; with pixel tiles innermost (order 1),
    // the reverse.
    const int64_t G = g.num_tiles, G8 = G & ~int64_t(7), per = G8 / 8;
    const double ker_slice = ker_line_bytes / g.tiles_k;
    std::vector<char> seen_px(tile_halo.size()), seen_k((size_t)g.tiles_k);
    double l2 = 0;
    auto take = [&](int64_t L) {
      int64_t kt, px;
      if (plan->grid_order == 0) {
        kt = L % g.tiles_k;
        px = L / g.tiles_k;
      } else {
        const int64_t ct = L % g.tiles_cols, rest = L / g.tiles_cols;
        kt = rest / g.tiles_rows;
        px = (rest % g.tiles_rows) * g.tiles_cols + ct;
      }
      if (!seen_px[(size_t)px]) seen_px[(size_t)px] = 1, l2 += tile_halo[(size_t)px];
      if (!seen_k[(size_t)kt]) seen_k[(size_t)kt] = 1, l2 += ker_slice;
    };
    for (int x = 0; x < 8; ++x) {
      std::fill(seen_px.begin(), seen_px.end(), 0);
      std::fill(seen_k.begin(), seen_k.end(), 0);
      for (int64_t L = x * per; L < (x + 1) * per; ++L) take(L);
      if (G8 + x < G) take(G8 + x);
    }
    plan->pred_bytes[CONV_LVL_L2] = l2;
    plan->class_lvl[CONV_LVL_L2] = plan->grid_order == 0 ? 5 : 1;
  } else if (plan->grid_order == 0) {
    // k tiles innermost: each pixel tile's halo is fetched once.  Every XCD
    // needs the whole kernel tensor; it stays resident if it fits in half the
    // XCD's L2, else it is re-fetched once per group of pixel tiles that are
    // in flight together on the XCD.
    double ker_l2;
    if (ker_bytes <= 0.5 * kHw.l2_bytes) {
      ker_l2 = std::min<double>(kHw.xcds, pix_tiles) * ker_line_bytes;
    } else {
      const double occ = std::max(1, std::min(2, kHw.lds_bytes / std::max(1, lds)));
      const double resident = (double)kHw.cus / kHw.xcds * occ;
      const double inflight = std::max(1.0, resident / g.tiles_k);
      ker_l2 = pix_tiles / inflight * ker_line_bytes;
    }
    plan->pred_bytes[CONV_LVL_L2] = in_halo_bytes + ker_l2;
    plan->class_lvl[CONV_LVL_L2] = 5;  // <{n,c,h,r,s}, w, k>: k innermost
  } else {
    // pixel tiles innermost: a k slice of Ker stays; In is re-read per k tile.
    plan->pred_bytes[CONV_LVL_L2] = in_halo_bytes * g.tiles_k + ker_line_bytes;
    plan->class_lvl[CONV_LVL_L2] = 1;  // <{k,c,r,s},{n,h},w>: pixels innermost
  }
  // split reduction: every range writes its partial Out to the workspace and
  // the second pass reads them all back
  const double ws_bytes = g.split > 1 ? 2.0 * g.split * out_bytes : 0.0;
  plan->pred_bytes[CONV_LVL_HBM] = in_bytes + ker_bytes + out_bytes + ws_bytes;
  plan->class_lvl[CONV_LVL_REG] = 3;  // <{n,k,h,w},{c,r},s>
  plan->class_lvl[CONV_LVL_LDS] = 3;
  plan->class_lvl[CONV_LVL_HBM] = 0;

  // Persistent kernels (bf16 families) give each workgroup a fixed run of
  // ceil(tiles / workgroups) tiles: the memory levels run at full rate only
  // while every workgroup still has tiles (the load-balancing term of
  // Algorithm 1 applied to the levels, not only to the MFMAs), and a tile
  // that the layer fills only in part (columns past Q, k rows past K) takes
  // a whole tile's phases; so the levels are charged the tile executions of
  // the busiest workgroup over the tiles' worth of useful outputs.  The last
  // tile's stores of every workgroup follow its MFMAs with nothing left to
  // overlap them.
  const bool persistent = v->family == FAMILY_BF16 || v->family == FAMILY_BF16_TR;
  double imbalance = 1.0, last_tile_us = kHw.drain_us;
  if (persistent && g.num_tiles > 0) {
    const double G = std::min<double>(g.grid, g.num_tiles);
    const double full = (double)g.num_tiles * g.tr * g.tw * 16.0 * v->wk * g.nwk /
                        ((double)s.N * g.P * g.Q * s.K);  // tile slots over outputs (>= 1)
    imbalance = std::ceil(g.num_tiles / G) * G / g.num_tiles * std::max(1.0, full);
    last_tile_us = G * (out_bytes / g.num_tiles) / kHw.bw[CONV_LVL_HBM] * 1e6;
  }
  double tmax = 0;
  for (int l = 0; l < CONV_NUM_LVLS; ++l) {
    plan->pred_us[l] = plan->pred_bytes[l] / kHw.bw[l] * 1e6;
    if (l == CONV_LVL_L2 || l == CONV_LVL_HBM) plan->pred_us[l] *= imbalance;
    tmax = std::max(tmax, plan->pred_us[l]);
  }
  // Compute: MFMA cycles of one wave (its channel range); a CU runs
  // ceil(workgroups / cus) workgroups whose waves share its SIMDs.
  const double mfma_per_step = (double)v->wk * v->wp;
  const double mfma_cycles = (plan->dtype == CONV_DTYPE_BF16) ? 16.0 : kHw.mfma_f32_cycles;
  const int groups = v->groups();
  const double wave_cycles = steps * ((double)g.cps / g.nchunks) * mfma_per_step * mfma_cycles / groups;
  // tile executions: grid = tiles x ranges, or fewer persistent workgroups
  const double per_cu = std::ceil((double)g.num_tiles * g.split / kHw.cus);
  const double waves_per_simd = per_cu * (g.nwk * g.nwp * groups) / kHw.simds_per_cu;
  plan->pred_mfma_us = waves_per_simd * wave_cycles / kHw.clock_hz * 1e6;
  // phase skip: the steps of zero taps are not run (3x3 stride 2: 9 of 16)
  if (v->phase_skip) plan->pred_mfma_us *= (2.0 * v->rc - 1) * (2.0 * v->sc - 1) / (4.0 * v->rc * v->sc);
  if (plan->dtype == CONV_DTYPE_F32) {
    // Issue efficiency of the fp32 inner loop.  Each step of a WK x WP wave
    // tile reads WK + WP operands from LDS for WK * WP MFMAs; measured
    // (inner-loop probes and layer sweeps on MI355X) the loop sustains about
    // c / (reads per MFMA) of the MFMA rate, capped: c = 0.53, cap 0.78 with
    // one wave per SIMD; c = 0.70, cap 0.82 when two or more waves share a
    // SIMD and cover each other's operand waits.
    const double reads_per_mfma = (double)(v->wk + v->wp) / ((double)v->wk * v->wp);
    const bool shared = (g.nwk * g.nwp * groups) > kHw.simds_per_cu;
    double eff = std::min(shared ? 0.82 : 0.78, (shared ? 0.70 : 0.53) / reads_per_mfma);
    // 32x32x2 loop: full-rate MFMAs from 4 accumulators on and fewer operand
    // reads per flop, yet measured on the 3x3 layers the MFMA pipe is busy
    // only about 55% of the time (busy counters; layer timings of the model
    // validation sweep), so it is scored at that efficiency
    if (v->mfma32) eff = 0.55;
    plan->pred_mfma_us /= eff;
  }
  tmax = std::max(tmax, plan->pred_mfma_us);
  // The reduction pass of a split plan runs after the main kernel: a launch
  // plus reading the ranges and writing Out.
  const double reduce_us =
      g.split > 1 ? kHw.launch_us + (g.split + 1.0) * out_bytes / kHw.bw[CONV_LVL_HBM] * 1e6 : 0.0;
  // Fill and drain: one round trip before the first step, that step's MFMAs
  // (nothing to overlap them with yet), the last stores.
  const double step_us = plan->pred_mfma_us / std::max(1, g.cps);
  plan->pred_total_us = tmax + reduce_us + kHw.fill_us + step_us + last_tile_us;
  return CONV_OK;
}

// Measured rate of each compiled kernel variant relative to the model
// (variant_calibration.inc, generated by paper_2101_09808_amd/calibrate.py
// from the rank sweep of the five layer configurations): the median over
// the variant's timed plans of measured / predicted time.  The model's
// levels and MFMA time do not capture how well an instance's inner loop
// hides latency and issues (the paper measures its microkernel's rate once,
// Sec. 6); this factor does, per instance.  A variant without enough timed
// plans takes its family's median; an unknown one 1.
#include "variant_calibration.inc"
struct Calibration {
  int id;  // variant id, or minus the family
  double factor;
  int plans;
};
const Calibration kCalibration[] = {CONV_CALIBRATION_TABLE};

double calibration(const Variant& v) {
  for (const Calibration& c : kCalibration)
    if (c.id == v.id) return c.factor;
  for (const Calibration& c : kCalibration)
    if (c.id == -v.family) return c.factor;
  return 1.0;
}

void fill_plan_fields(conv_plan_t* p, const Variant& v, int nwk, int nwp, int tr, int tw,
                      int order) {
  std::memset(p, 0, sizeof(*p));
  p->dtype = v.dtype;
  p->variant = v.id;
  p->tile_k = 16 * v.wk * nwk;
  p->tile_rows = tr;
  p->tile_cols = tw;
  p->tile_c = v.tc;
  p->wave_k = 16 * v.wk;
  p->wave_px = 16 * v.wp;
  p->waves_k = nwk;
  p->waves_px = nwp;
  p->grid_order = order;
  p->split_c = 1;
}

// Deterministic preference among plans (tie-breaks: predicted time times
// the family factor, MFMA time, total predicted bytes, fewer workgroups,
// variant id, larger k tile, no split).
bool better(const conv_plan_t& a, const conv_plan_t& b) {
  const double ta = rank_time(a), tb = rank_time(b);
  if (ta != tb) return ta < tb;
  // equal bound: less MFMA work (fewer padded pixels in partial tiles)
  if (a.pred_mfma_us != b.pred_mfma_us) return a.pred_mfma_us < b.pred_mfma_us;
  double ba = 0, bb = 0;
  for (int l = 0; l < CONV_NUM_LVLS; ++l) {
    ba += a.pred_bytes[l];
    bb += b.pred_bytes[l];
  }
  if (ba != bb) return ba < bb;
  if (a.num_wg != b.num_wg) return a.num_wg < b.num_wg;
  if (a.variant != b.variant) return a.variant < b.variant;
  if (a.tile_k != b.tile_k) return a.tile_k > b.tile_k;
  if (a.tile_rows != b.tile_rows) return a.tile_rows > b.tile_rows;
  if (a.tile_cols != b.tile_cols) return a.tile_cols > b.tile_cols;
  if (a.grid_order != b.grid_order) return a.grid_order < b.grid_order;
  return a.split_c < b.split_c;
}
}  // namespace

int enumerate_plans(const Shape& s0, int dtype, conv_plan_t* plans, int cap, bool phase_skip) {
  const Shape s = kernel_view(s0);
  int nv = 0;
  const Variant* vs = variants(&nv);
  std::vector<conv_plan_t> all;
  const int P = s.P(), Q = s.Q();
  for (int vi = 0; vi < nv; ++vi) {
    const Variant& v = vs[vi];
    if (v.dtype != dtype) continue;
    if (v.phase_skip && !phase_skip) continue;  // only for conv_fwd_ex's stride-2 odd-tap layers
    if (v.rc && (s.R != v.rc || s.S != v.sc)) continue;
    if (v.family == FAMILY_STREAM1X1 || v.family == FAMILY_STREAM1X1_LOOP) {
      // pixels per wave so that the workgroup count lands near a multiple
      // of the CU count; the instance's block count must match
      const int nb = v.wp;
      const int64_t total_px = (int64_t)s.N * s.W;
      std::vector<int> wpxs;
      for (int64_t G = 1; G <= 4096; ++G) {
        const int64_t wpx = cdiv(total_px, 4 * G);
        if (wpx > 16 * (nb - 1) && wpx <= 16 * nb &&
            std::find(wpxs.begin(), wpxs.end(), (int)wpx) == wpxs.end())
          wpxs.push_back((int)wpx);
      }
      if (wpxs.empty() && 16 * nb >= cdiv(total_px, 4)) wpxs.push_back((int)cdiv(total_px, 4));
      for (int wpx : wpxs) {
        conv_plan_t p;
        fill_plan_fields(&p, v, 1, 4, 1, wpx, 0);
        p.tile_k = 64;
        p.wave_k = 64;
        if (score_plan(s0, &p) == CONV_OK) all.push_back(p);
      }
      continue;
    }
    if (v.family == FAMILY_STREAM1X1_BAL) {
      // pixels per workgroup: every share that leaves NB whole blocks per
      // wave and at most 16 pixels for the k-split tail block
      const int nb = v.max_ni;
      const int64_t total_px = (int64_t)s.N * s.W;
      std::vector<int> pws;
      for (int64_t G = cdiv(total_px, 128 * nb + 16); G <= 65536; ++G) {
        const int64_t pw = cdiv(total_px, G);
        if (pw <= 128 * nb) break;
        if (pw <= 128 * nb + 16 && std::find(pws.begin(), pws.end(), (int)pw) == pws.end())
          pws.push_back((int)pw);
      }
      for (int pw : pws) {
        conv_plan_t p;
        fill_plan_fields(&p, v, 1, 4, 1, pw, 0);
        p.tile_k = 64;
        p.wave_k = 64;
        if (score_plan(s0, &p) == CONV_OK) all.push_back(p);
      }
      continue;
    }
    // Four channels per step only for layers with few channels (a first
    // layer, a stride-2 7x7 layer's 12 phase channels), where a wider step
    // is mostly zeros; elsewhere the extra pipeline steps cost more than
    // they save (3x3 N32 C128: 100 us at four channels per step, 93 us at
    // eight).
    if (v.family == FAMILY_DMA && v.tc < 8 && s.C >= 16) continue;
    const int nw = v.threads / 64 / v.groups();  // waves per channel group
    for (int nwk = 1; nwk <= nw; ++nwk) {
      if (nw % nwk) continue;
      const int nwp = nw / nwk;
      const int BP = 16 * v.wp * nwp;
      // Column tiles: whole rows, or Q split into m near-equal parts (the
      // transposing bf16 kernel: multiples of 16, rows filling the blocks).
      std::vector<int> tws;
      if (v.family == FAMILY_BF16_TR) {
        tws.push_back(v.max_nk);  // compile-time tile
      } else {
        for (int m = 1; m <= 16; ++m) {
          const int tw = (int)cdiv(Q, m);
          if (tw <= BP && std::find(tws.begin(), tws.end(), tw) == tws.end()) tws.push_back(tw);
        }
        if (Q > BP) tws.push_back(BP);
      }
      for (int tw : tws) {
        const int tr_max = v.family == FAMILY_BF16_TR ? v.max_ni : BP / tw;
        // Row tiles: as many rows as fit, or a divisor-friendly smaller count.
        std::vector<int> trs = {tr_max};
        if (tr_max > 1 && P % tr_max) {
          for (int d = tr_max - 1; d >= 1; --d)
            if (P % d == 0 || d % P == 0) {
              trs.push_back(d);
              break;
            }
        }
        for (int tr : trs)
          for (int order = 0; order < 2; ++order) {
            conv_plan_t p;
            fill_plan_fields(&p, v, nwk, nwp, tr, tw, order);
            if (score_plan(s0, &p) != CONV_OK) continue;
            // Channel groups of waves pay the pipeline's fill and the LDS
            // reduction once per workgroup, with one workgroup per CU: they
            // are for grids that fit the CUs in one round (measured on
            // MI355X, they win there and lose up to 1.8x on larger grids),
            // and they replace the split reduction rather than add to it
            // (each split measured slower than the same plan unsplit).
            if (v.groups() > 1 && p.num_wg > kHw.cus) continue;
            all.push_back(p);
            // Too few workgroups to fill the CUs: also split the channel
            // reduction into ranges (direct-to-LDS kernel only).
            if (v.family == FAMILY_DMA && v.groups() == 1 && p.num_wg < kHw.cus) {
              for (int split : {2, 3, 4, 6, 8, 12, 16}) {
                if (p.num_wg * split > 2 * kHw.cus) break;
                conv_plan_t q = p;
                q.split_c = split;
                if (score_plan(s0, &q) == CONV_OK) all.push_back(q);
              }
            }
          }
      }
    }
  }
  std::sort(all.begin(), all.end(), better);
  const int n = (int)all.size();
  for (int i = 0; i < n && i < cap; ++i) plans[i] = all[i];
  return n;
}

int select_plan(const Shape& s, int dtype, conv_plan_t* out) {
  std::vector<conv_plan_t> buf(4096);
  const int n = enumerate_plans(s, dtype, buf.data(), (int)buf.size());
  if (n <= 0) return CONV_ENOPLAN;
  *out = buf[0];
  return CONV_OK;
}

}  // namespace convfwd
