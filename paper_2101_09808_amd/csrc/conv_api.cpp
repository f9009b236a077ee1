// C ABI of the convolution library: argument validation, the per-shape plan
// cache and dispatch to the kernels.  The declarations and their contracts
// are in include/conv_fwd.h.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <map>
#include <mutex>
#include <tuple>
#include <vector>

#include "conv_internal.h"

using namespace convfwd;

namespace {

const int64_t kMaxElems = (int64_t(1) << 31) - 1;

int validate_shape(int N, int C, int K, int H, int W, int R, int S) {
  if (N <= 0 || C <= 0 || K <= 0 || H <= 0 || W <= 0 || R <= 0 || S <= 0) return CONV_EINVAL;
  if (R > H || S > W) return CONV_EINVAL;
  const int64_t P = H - R + 1, Q = W - S + 1;
  if ((int64_t)N * C * H * W > kMaxElems) return CONV_ERANGE;
  if ((int64_t)K * C * R * S > kMaxElems) return CONV_ERANGE;
  if ((int64_t)N * K * P * Q > kMaxElems) return CONV_ERANGE;
  return CONV_OK;
}

// Per (shape, dtype, tensor alignment) the selected plan and its resolved launch.
struct Entry {
  conv_plan_t plan;
  const Variant* v;
  Geom g;
};
typedef std::tuple<int, int, int, int, int, int, int, int, int> Key;
std::mutex g_mu;
std::map<Key, Entry> g_cache;

// Alignment bits of a call: vector loads of In (4 fp32) or Ker need a
// 16-byte aligned tensor; the transposing bf16 kernel loads In in dwords.
enum { ALIGN_KER = 1, ALIGN_IN = 2, ALIGN_IN4 = 4, ALIGN_ALL = 7 };

int alignment_of(const void* In, const void* Ker) {
  return ((reinterpret_cast<uintptr_t>(Ker) & 15) == 0 ? ALIGN_KER : 0) |
         ((reinterpret_cast<uintptr_t>(In) & 15) == 0 ? ALIGN_IN : 0) |
         ((reinterpret_cast<uintptr_t>(In) & 3) == 0 ? ALIGN_IN4 : 0);
}

// Does variant v run with tensors of this alignment?
bool variant_fits(const Variant& v, int dtype, int align) {
  const int elem = dtype == CONV_DTYPE_BF16 ? 2 : 4;
  if (v.ker_vec * elem > elem && v.family != FAMILY_BF16 && !(align & ALIGN_KER)) return false;
  if (v.family == FAMILY_DMA && v.in_vec > 1 && !(align & ALIGN_IN)) return false;
  if (v.family == FAMILY_BF16_TR && !(align & ALIGN_IN4)) return false;
  return true;
}

int select_entry(const Shape& s, int dtype, int align, Entry* e) {
  conv_plan_t p;
  int st = select_plan(s, dtype, &p);
  if (st != CONV_OK) return st;
  const Variant* v = find_variant(p.variant);
  if (v && !variant_fits(*v, dtype, align)) {
    // best plan of a variant whose loads suit the tensors' alignment
    std::vector<conv_plan_t> buf(4096);
    const int n = enumerate_plans(s, dtype, buf.data(), (int)buf.size());
    v = nullptr;
    for (int i = 0; i < n && i < (int)buf.size(); ++i) {
      const Variant* w = find_variant(buf[i].variant);
      if (w && variant_fits(*w, dtype, align)) {
        p = buf[i];
        v = w;
        break;
      }
    }
    if (!v) return CONV_ENOPLAN;
  }
  if (!v || !resolve_geom(s, *v, p, &e->g, nullptr)) return CONV_ENOPLAN;
  e->plan = p;
  e->v = v;
  return CONV_OK;
}

int cached_entry(const Shape& s, int dtype, int align, Entry* out) {
  const Key key{s.N, s.C, s.K, s.H, s.W, s.R, s.S, dtype, align};
  {
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_cache.find(key);
    if (it != g_cache.end()) {
      *out = it->second;
      return CONV_OK;
    }
  }
  Entry e;
  const int st = select_entry(s, dtype, align, &e);
  if (st != CONV_OK) return st;
  {
    std::lock_guard<std::mutex> lk(g_mu);
    g_cache[key] = e;
  }
  *out = e;
  return CONV_OK;
}

// bf16 Out from the transposing bf16 kernel: its stores are 16 bytes only
// when the wave tile pairs neighbouring blocks (an even number of blocks per
// part, in rows of an even number of blocks); otherwise every output is a
// 2-byte store, eight times slower on the 226x226 layer.  Whether a tile
// pairs is fixed by the instance (rows max_ni, columns max_nk), as in the
// kernel's PAIRED.
bool pairs_bf16_out(const Variant& v) {
  if (v.family != FAMILY_BF16_TR) return true;
  const int cbr = v.max_nk / 16, wp = v.max_ni * cbr / 4;
  const int npart = wp % 2 == 0 ? 2 : 1, pb = wp / npart;
  return pb % 2 == 0 && cbr % 2 == 0;
}

// The plan of conv_fwd_bf16_out: the selected bf16 plan, unless 16-byte
// stores are possible (Q % 8 == 0, Out 16-byte aligned) and it does not pair
// them: then the best candidate that does.  Cached beside the other entries
// under its own dtype code.
constexpr int kBf16OutKey = 0x100;
int cached_entry_bf16_out(const Shape& s, int align, bool pair_possible, Entry* out) {
  Entry e;
  int st = cached_entry(s, CONV_DTYPE_BF16, align, &e);
  if (st != CONV_OK || !pair_possible || pairs_bf16_out(*e.v)) {
    *out = e;
    return st;
  }
  const Key key{s.N, s.C, s.K, s.H, s.W, s.R, s.S, CONV_DTYPE_BF16 | kBf16OutKey, align};
  {
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_cache.find(key);
    if (it != g_cache.end()) {
      *out = it->second;
      return CONV_OK;
    }
  }
  std::vector<conv_plan_t> buf(4096);
  const int n = std::min<int>(enumerate_plans(s, CONV_DTYPE_BF16, buf.data(), (int)buf.size()), (int)buf.size());
  for (int i = 0; i < n; ++i) {
    const Variant* w = find_variant(buf[i].variant);
    Geom g;
    if (!w || !variant_fits(*w, CONV_DTYPE_BF16, align) || !pairs_bf16_out(*w) ||
        !resolve_geom(s, *w, buf[i], &g, nullptr))
      continue;
    e.plan = buf[i];
    e.v = w;
    e.g = g;
    break;
  }
  {
    std::lock_guard<std::mutex> lk(g_mu);
    g_cache[key] = e;
  }
  *out = e;
  return CONV_OK;
}

int cached_plan(const Shape& s, int dtype, conv_plan_t* out) {
  Entry e;
  const int st = cached_entry(s, dtype, ALIGN_ALL, &e);
  if (st == CONV_OK) *out = e.plan;
  return st;
}

int run(const Shape& s, const void* In, const void* Ker, float* Out, const conv_plan_t& plan,
        void* stream) {
  const Variant* v = find_variant(plan.variant);
  if (!v || v->dtype != plan.dtype || v->phase_skip) return CONV_EINVAL;  // phase skip: conv_fwd_ex only
  if (!variant_fits(*v, plan.dtype, alignment_of(In, Ker))) return CONV_EINVAL;
  Geom g;
  if (!resolve_geom(s, *v, plan, &g, nullptr)) return CONV_EINVAL;
  return launch(*v, g, In, Ker, Out, stream);
}

// Selected plan for a call: cached per shape and tensor alignment.
// bf16 shapes that no bf16 kernel instance takes (other tap counts): the
// inputs are widened exactly to fp32 in a stream-ordered workspace and the
// fp32 plan runs -- the same products and fp32 sums.  out_bf16: Out is
// bf16, written by rounding an fp32 result kept in the workspace.
int run_bf16_widened(const Shape& s, const void* In, const void* Ker, void* Out, bool out_bf16, void* stream) {
  const size_t n_in = (size_t)s.N * s.C * s.H * s.W, n_ker = (size_t)s.K * s.C * s.R * s.S;
  const size_t n_out = out_bf16 ? (size_t)s.N * s.K * (s.H - s.R + 1) * (s.W - s.S + 1) : 0;
  const size_t a_in = (n_in * 4 + 255) / 256 * 256, a_ker = (n_ker * 4 + 255) / 256 * 256;
  Workspace w;
  int st = workspace_acquire(0, a_in + a_ker + n_out * 4, stream, &w);
  if (st != CONV_OK) return st;
  void* ws = w.ptr;
  float* in32 = static_cast<float*>(ws);
  float* ker32 = reinterpret_cast<float*>(static_cast<char*>(ws) + a_in);
  float* out32 = reinterpret_cast<float*>(static_cast<char*>(ws) + a_in + a_ker);
  st = launch_widen_bf16(In, in32, (int64_t)n_in, stream);
  if (st == CONV_OK) st = launch_widen_bf16(Ker, ker32, (int64_t)n_ker, stream);
  if (st == CONV_OK) {
    Entry e;
    st = cached_entry(s, CONV_DTYPE_F32, alignment_of(in32, ker32), &e);
    if (st == CONV_OK) st = launch(*e.v, e.g, in32, ker32, out_bf16 ? out32 : static_cast<float*>(Out), stream);
  }
  if (st == CONV_OK && out_bf16) st = launch_round_bf16(out32, Out, (int64_t)n_out, stream);
  const int freed = workspace_release(w, stream);
  return st == CONV_OK ? freed : st;
}

int run_selected(const Shape& s, int dtype, const void* In, const void* Ker, float* Out,
                 void* stream) {
  Entry e;
  const int st = cached_entry(s, dtype, alignment_of(In, Ker), &e);
  if (st == CONV_ENOPLAN && dtype == CONV_DTYPE_BF16) return run_bf16_widened(s, In, Ker, Out, false, stream);
  if (st != CONV_OK) return st;
  return launch(*e.v, e.g, In, Ker, Out, stream);
}

// conv_fwd_ex's plan for an fp32 strided or padded layer: the selector's
// plan of the inner problem (the best one whose loads suit the tensors as
// the kernel will see them), run reading In through the phase mapping when
// its kernel can.  Cached per layer, stride, padding and alignment.
struct ExEntry {
  Entry e;
  bool direct;  // e.g carries the phase mapping
};
typedef std::tuple<int, int, int, int, int, int, int, int, int, int, int, int> ExKey;
std::map<ExKey, ExEntry> g_ex_cache;

int select_ex_entry(const PhaseGeom& p, int align_direct, int align_split, ExEntry* out) {
  const Shape inner{p.N, p.C * p.na * p.nb, p.K, p.Hp, p.Wp, p.Rp, p.Sp};
  // (Ranking the candidates with the phase-split pass charged to plans that
  // cannot read In directly picked worse plans on the small layers, whose
  // predicted times are least reliable: Table 1's R1 28 -> 54 us.)
  // Stride-2 layers with odd taps also get the phase-skip variants, which
  // run only reading In directly.
  const bool skip_ok = p.na == 2 && p.nb == 2 && p.sh == 2 && p.sw == 2 && p.R == 2 * p.Rp - 1 &&
                       p.S == 2 * p.Sp - 1;
  std::vector<conv_plan_t> buf(4096);
  const int n =
      std::min<int>(enumerate_plans(inner, CONV_DTYPE_F32, buf.data(), (int)buf.size(), skip_ok), (int)buf.size());
  for (int i = 0; i < n; ++i) {
    const Variant* v = find_variant(buf[i].variant);
    Geom g;
    if (!v || !resolve_geom(inner, *v, buf[i], &g, nullptr)) continue;
    Geom gd = g;
    const bool direct = variant_fits(*v, CONV_DTYPE_F32, align_direct) && phase_direct(*v, p, CONV_DTYPE_F32, &gd);
    if (v->phase_skip && !direct) continue;
    if (!direct && !variant_fits(*v, CONV_DTYPE_F32, align_split)) continue;
    out->e.plan = buf[i];
    out->e.v = v;
    out->e.g = direct ? gd : g;
    out->direct = direct;
    return CONV_OK;
  }
  return CONV_ENOPLAN;
}

int cached_ex_entry(const PhaseGeom& p, int align_direct, int align_split, ExEntry* out) {
  const ExKey key{p.N, p.C, p.K, p.H, p.W, p.R, p.S, p.sh, p.sw, p.ph, p.pw, align_direct * 8 + align_split};
  {
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_ex_cache.find(key);
    if (it != g_ex_cache.end()) {
      *out = it->second;
      return CONV_OK;
    }
  }
  ExEntry e;
  const int st = select_ex_entry(p, align_direct, align_split, &e);
  if (st != CONV_OK) return st;
  std::lock_guard<std::mutex> lk(g_mu);
  g_ex_cache[key] = e;
  *out = e;
  return CONV_OK;
}

// Inner stride-1 problem of a strided, padded convolution (polyphase rewrite).
int phase_geom(int N, int C, int K, int H, int W, int R, int S, int sh, int sw, int ph, int pw,
               PhaseGeom* p) {
  if (N <= 0 || C <= 0 || K <= 0 || H <= 0 || W <= 0 || R <= 0 || S <= 0) return CONV_EINVAL;
  if (sh < 1 || sw < 1 || ph < 0 || pw < 0 || sh > 64 || sw > 64 || ph > 4096 || pw > 4096) return CONV_EINVAL;
  if (H + 2 * ph < R || W + 2 * pw < S) return CONV_EINVAL;
  PhaseGeom q;
  q.N = N; q.C = C; q.K = K; q.H = H; q.W = W; q.R = R; q.S = S;
  q.sh = sh; q.sw = sw; q.ph = ph; q.pw = pw;
  q.P = (H + 2 * ph - R) / sh + 1;
  q.Q = (W + 2 * pw - S) / sw + 1;
  q.na = std::min(sh, R);
  q.nb = std::min(sw, S);
  q.Rp = (R + sh - 1) / sh;
  q.Sp = (S + sw - 1) / sw;
  q.Hp = q.P + q.Rp - 1;
  q.Wp = q.Q + q.Sp - 1;
  if ((int64_t)C * q.na * q.nb > kMaxElems) return CONV_ERANGE;
  const int st = validate_shape(N, C * q.na * q.nb, K, q.Hp, q.Wp, q.Rp, q.Sp);
  if (st != CONV_OK) return st;
  if ((int64_t)N * C * H * W > kMaxElems) return CONV_ERANGE;
  *p = q;
  return CONV_OK;
}

// The fields of conv_fwd_geometry, in the header's order.
int export_geometry(const Variant& vr, const Geom& g, int lds, int32_t* out, int cap) {
  const Variant* v = &vr;
  const int32_t f[CONV_GEOM_FIELDS] = {
      g.N, g.C, g.K, g.H, g.W, g.R, g.S, g.P, g.Q,
      g.tr, g.tw, g.tiles_rows, g.tiles_cols, g.tiles_k,
      g.in_rows, g.in_wp, g.in_cstride, g.ker_rstride,
      g.nwk, g.nwp, g.order, g.num_tiles,
      g.lds_in_elems, g.lds_ker_elems, g.ni_in, g.ni_ker, g.nchunks,
      v->wk, v->wp, v->tc, v->rc, v->sc, v->max_ni, v->max_nk, v->ker_vec, v->threads, lds,
      v->family, v->in_vec, v->stages, g.stage_elems, g.in_region, (int32_t)g.in_bytes,
      (int32_t)g.ker_bytes, g.grid, v->phase_skip, 0, 0, g.split, g.cps, v->mfma32, v->groups(),
      g.nph, g.na, g.nb, g.sh, g.sw, g.ph, g.pw, g.C0, g.H0, g.W0, g.Wi,
      (int32_t)g.dv_in_cstride.m, g.dv_in_cstride.s, (int32_t)g.dv_in_wp.m, g.dv_in_wp.s,
      (int32_t)g.dv_H.m, g.dv_H.s, (int32_t)g.dv_ker_rstride.m, g.dv_ker_rstride.s,
      (int32_t)g.dv_tw.m, g.dv_tw.s, (int32_t)g.dv_P.m, g.dv_P.s, (int32_t)g.dv_nph.m, g.dv_nph.s,
      (int32_t)g.dv_nb.m, g.dv_nb.s, (int32_t)g.dv_Wi.m, g.dv_Wi.s, (int32_t)g.dv_tiles_k.m, g.dv_tiles_k.s,
      (int32_t)g.dv_tiles_cols.m, g.dv_tiles_cols.s, (int32_t)g.dv_tiles_rows.m, g.dv_tiles_rows.s};
  for (int i = 0; i < cap && i < CONV_GEOM_FIELDS; ++i) out[i] = f[i];
  return CONV_GEOM_FIELDS;
}

}  // namespace

extern "C" {

int conv_fwd(int N, int C, int K, int H, int W, int R, int S, const float* In, const float* Ker,
             float* Out, void* stream) {
  int st = validate_shape(N, C, K, H, W, R, S);
  if (st != CONV_OK) return st;
  if (!In || !Ker || !Out) return CONV_ENULL;
  return run_selected(Shape{N, C, K, H, W, R, S}, CONV_DTYPE_F32, In, Ker, Out, stream);
}

int conv_fwd_bf16(int N, int C, int K, int H, int W, int R, int S, const uint16_t* In,
                  const uint16_t* Ker, float* Out, void* stream) {
  int st = validate_shape(N, C, K, H, W, R, S);
  if (st != CONV_OK) return st;
  if (!In || !Ker || !Out) return CONV_ENULL;
  return run_selected(Shape{N, C, K, H, W, R, S}, CONV_DTYPE_BF16, In, Ker, Out, stream);
}

int conv_fwd_bf16_out(int N, int C, int K, int H, int W, int R, int S, const uint16_t* In,
                      const uint16_t* Ker, uint16_t* Out, void* stream) {
  int st = validate_shape(N, C, K, H, W, R, S);
  if (st != CONV_OK) return st;
  if (!In || !Ker || !Out) return CONV_ENULL;
  Entry e;
  const Shape sh{N, C, K, H, W, R, S};
  const bool pair_possible = (W - S + 1) % 8 == 0 && (reinterpret_cast<uintptr_t>(Out) & 15) == 0;
  st = cached_entry_bf16_out(sh, alignment_of(In, Ker), pair_possible, &e);
  if (st == CONV_ENOPLAN) return run_bf16_widened(sh, In, Ker, Out, true, stream);
  if (st != CONV_OK) return st;
  return launch_bf16_out(*e.v, e.g, In, Ker, Out, stream);
}

}  // extern "C"

namespace {

// The body of conv_fwd_ex (arguments already validated).
int run_ex(const PhaseGeom& p, int dtype, const void* In, const void* Ker, float* Out, void* stream) {
  const int N = p.N, C = p.C, K = p.K, H = p.H, W = p.W, R = p.R, S = p.S;
  int st = CONV_OK;
  if (p.sh == 1 && p.sw == 1 && p.ph == 0 && p.pw == 0)
    return run_selected(Shape{N, C, K, H, W, R, S}, dtype, In, Ker, static_cast<float*>(Out), stream);
  const size_t e = dtype == CONV_DTYPE_BF16 ? 2 : 4;
  const int Cp = C * p.na * p.nb;
  // The rearranged Ker differs from Ker only with more than one phase (one
  // phase per axis means stride 1 or a single tap along it).
  const bool ker_moves = p.na * p.nb > 1;
  const Shape inner{N, Cp, K, p.Hp, p.Wp, p.Rp, p.Sp};
  if (dtype == CONV_DTYPE_F32) {
    // The plan either reads the caller's In through the phase mapping
    // (direct-to-LDS kernel: no pass over In) or runs on phase-split copies
    // in a workspace; a strided Ker is rearranged first either way.  The
    // workspaces are 256-byte aligned.
    const int ker_al = ker_moves ? ALIGN_KER : (alignment_of(In, Ker) & ALIGN_KER);
    const int al_direct = (alignment_of(In, Ker) & (ALIGN_IN | ALIGN_IN4)) | ker_al;
    const int al_split = ALIGN_IN | ALIGN_IN4 | ker_al;
    ExEntry x;
    st = cached_ex_entry(p, al_direct, al_split, &x);
    if (st != CONV_OK) return st;
    const size_t in_ws = x.direct ? 0 : ((size_t)N * Cp * p.Hp * p.Wp * e + 255) / 256 * 256;
    const size_t ker_ws = ker_moves ? (size_t)K * Cp * p.Rp * p.Sp * e : 0;
    if (in_ws + ker_ws == 0) return launch(*x.e.v, x.e.g, In, Ker, Out, stream);
    Workspace w;
    st = workspace_acquire(0, in_ws + ker_ws, stream, &w);
    if (st != CONV_OK) return st;
    char* ws = static_cast<char*>(w.ptr);
    void* Kp = ker_moves ? ws + in_ws : nullptr;
    st = launch_phase_split(p, dtype, In, Ker, x.direct ? nullptr : ws, Kp, stream);
    if (st == CONV_OK)
      st = launch(*x.e.v, x.e.g, x.direct ? In : ws, ker_moves ? Kp : Ker, Out, stream);
    const int freed = workspace_release(w, stream);
    return st == CONV_OK ? freed : st;
  }
  // bf16: stream-ordered workspace with the phase images of In, then
  // (strided only) the rearranged Ker; at stride 1 the padded In meets the
  // original Ker
  const size_t in_bytes = ((size_t)N * Cp * p.Hp * p.Wp * e + 255) / 256 * 256;
  const size_t ker_bytes = ker_moves ? (size_t)K * Cp * p.Rp * p.Sp * e : 0;
  Workspace w;
  st = workspace_acquire(0, in_bytes + ker_bytes, stream, &w);
  if (st != CONV_OK) return st;
  char* ws = static_cast<char*>(w.ptr);
  void* Kp = ker_moves ? ws + in_bytes : nullptr;
  st = launch_phase_split(p, dtype, In, Ker, ws, Kp, stream);
  if (st == CONV_OK)
    st = run_selected(inner, dtype, ws, ker_moves ? Kp : Ker, Out, stream);
  const int freed = workspace_release(w, stream);
  return st == CONV_OK ? freed : st;
}

// Scratch bytes run_ex needs for these arguments, summed over the
// workspaces it takes in order, each rounded up to the 256-byte alignment
// of the arena's bump allocation.  Mirrors the dispatch of run_ex,
// run_selected, run_bf16_widened and launch (split partial sums); any
// workspace the library carves is 256-byte aligned, which is what the
// alignment of the plans that run on workspaces is computed with.
size_t up256(size_t b) { return (b + 255) / 256 * 256; }

size_t split_need(const Geom& g) {
  return g.split > 1 ? up256((size_t)g.split * g.N * g.K * g.P * g.Q * sizeof(float)) : 0;
}

int selected_need(const Shape& s, int dtype, int align, size_t* need) {
  Entry e;
  int st = cached_entry(s, dtype, align, &e);
  if (st == CONV_ENOPLAN && dtype == CONV_DTYPE_BF16) {
    // run_bf16_widened: exact fp32 copies of In and Ker, then the fp32 plan
    const size_t n_in = (size_t)s.N * s.C * s.H * s.W, n_ker = (size_t)s.K * s.C * s.R * s.S;
    const size_t wide = up256(up256(n_in * 4) + up256(n_ker * 4));
    st = cached_entry(s, CONV_DTYPE_F32, ALIGN_ALL, &e);
    if (st != CONV_OK) return st;
    *need = wide + split_need(e.g);
    return CONV_OK;
  }
  if (st != CONV_OK) return st;
  *need = split_need(e.g);
  return CONV_OK;
}

int ex_need(const PhaseGeom& p, int dtype, const void* In, const void* Ker, size_t* need) {
  const Shape s{p.N, p.C, p.K, p.H, p.W, p.R, p.S};
  if (p.sh == 1 && p.sw == 1 && p.ph == 0 && p.pw == 0) return selected_need(s, dtype, alignment_of(In, Ker), need);
  const size_t e = dtype == CONV_DTYPE_BF16 ? 2 : 4;
  const int Cp = p.C * p.na * p.nb;
  const bool ker_moves = p.na * p.nb > 1;
  const Shape inner{p.N, Cp, p.K, p.Hp, p.Wp, p.Rp, p.Sp};
  if (dtype == CONV_DTYPE_F32) {
    const int ker_al = ker_moves ? ALIGN_KER : (alignment_of(In, Ker) & ALIGN_KER);
    const int al_direct = (alignment_of(In, Ker) & (ALIGN_IN | ALIGN_IN4)) | ker_al;
    const int al_split = ALIGN_IN | ALIGN_IN4 | ker_al;
    ExEntry x;
    const int st = cached_ex_entry(p, al_direct, al_split, &x);
    if (st != CONV_OK) return st;
    const size_t in_ws = x.direct ? 0 : up256((size_t)p.N * Cp * p.Hp * p.Wp * e);
    const size_t ker_ws = ker_moves ? (size_t)p.K * Cp * p.Rp * p.Sp * e : 0;
    *need = (in_ws + ker_ws ? up256(in_ws + ker_ws) : 0) + split_need(x.e.g);
    return CONV_OK;
  }
  const size_t in_bytes = up256((size_t)p.N * Cp * p.Hp * p.Wp * e);
  const size_t ker_bytes = ker_moves ? (size_t)p.K * Cp * p.Rp * p.Sp * e : 0;
  // the inner plan runs on the (aligned) phase images and the rearranged or
  // the caller's Ker
  const int align = ALIGN_IN | ALIGN_IN4 | (ker_moves ? ALIGN_KER : (alignment_of(In, Ker) & ALIGN_KER));
  size_t inner_need = 0;
  const int st = selected_need(inner, dtype, align, &inner_need);
  if (st != CONV_OK) return st;
  *need = up256(in_bytes + ker_bytes) + inner_need;
  return CONV_OK;
}

// Installs an arena on the calling thread for the lifetime of the guard.
struct ArenaGuard {
  explicit ArenaGuard(ScratchArena* a) { set_thread_arena(a); }
  ~ArenaGuard() { set_thread_arena(nullptr); }
};

}  // namespace

extern "C" {

int conv_fwd_ex(int N, int C, int K, int H, int W, int R, int S, int stride_h, int stride_w, int pad_h,
                int pad_w, int dtype, const void* In, const void* Ker, float* Out, void* stream) {
  PhaseGeom p;
  const int st = phase_geom(N, C, K, H, W, R, S, stride_h, stride_w, pad_h, pad_w, &p);
  if (st != CONV_OK) return st;
  if (!In || !Ker || !Out) return CONV_ENULL;
  if (dtype != CONV_DTYPE_F32 && dtype != CONV_DTYPE_BF16) return CONV_EINVAL;
  return run_ex(p, dtype, In, Ker, Out, stream);
}

int conv_fwd_ex_noalloc(int N, int C, int K, int H, int W, int R, int S, int stride_h, int stride_w, int pad_h,
                        int pad_w, int dtype, const void* In, const void* Ker, float* Out, void* stream) {
  PhaseGeom p;
  int st = phase_geom(N, C, K, H, W, R, S, stride_h, stride_w, pad_h, pad_w, &p);
  if (st != CONV_OK) return st;
  if (!In || !Ker || !Out) return CONV_ENULL;
  if (dtype != CONV_DTYPE_F32 && dtype != CONV_DTYPE_BF16) return CONV_EINVAL;
  size_t need = 0;
  st = ex_need(p, dtype, In, Ker, &need);
  if (st != CONV_OK) return st;
  if (need > (size_t)CONV_NOALLOC_SCRATCH_BYTES) return CONV_ESCRATCH;
  void* base = nullptr;
  if (need > 0) {
    st = noalloc_scratch(&base);
    if (st != CONV_OK) return st;
  }
  ScratchArena arena{static_cast<char*>(base), need > 0 ? (size_t)CONV_NOALLOC_SCRATCH_BYTES : 0, 0};
  ArenaGuard guard(&arena);
  return run_ex(p, dtype, In, Ker, Out, stream);
}

int conv_fwd_ex_plan(int N, int C, int K, int H, int W, int R, int S, int stride_h, int stride_w, int pad_h,
                     int pad_w, int dtype, conv_plan_t* plan_out, int32_t* direct) {
  PhaseGeom p;
  int st = phase_geom(N, C, K, H, W, R, S, stride_h, stride_w, pad_h, pad_w, &p);
  if (st != CONV_OK) return st;
  if (!plan_out) return CONV_ENULL;
  if (dtype != CONV_DTYPE_F32 && dtype != CONV_DTYPE_BF16) return CONV_EINVAL;
  const bool rewrite = stride_h > 1 || stride_w > 1 || pad_h > 0 || pad_w > 0;
  if (dtype == CONV_DTYPE_F32 && rewrite) {
    ExEntry x;
    st = cached_ex_entry(p, ALIGN_ALL, ALIGN_ALL, &x);
    if (st != CONV_OK) return st;
    *plan_out = x.e.plan;
    if (direct) *direct = x.direct ? 1 : 0;
    return CONV_OK;
  }
  if (direct) *direct = 0;
  return cached_plan(Shape{N, C * p.na * p.nb, K, p.Hp, p.Wp, p.Rp, p.Sp}, dtype, plan_out);
}

int conv_fwd_ex_inner_shape(int N, int C, int K, int H, int W, int R, int S, int stride_h, int stride_w,
                            int pad_h, int pad_w, int32_t inner[9]) {
  if (!inner) return CONV_ENULL;
  PhaseGeom p;
  const int st = phase_geom(N, C, K, H, W, R, S, stride_h, stride_w, pad_h, pad_w, &p);
  if (st != CONV_OK) return st;
  const int32_t v[9] = {N, C * p.na * p.nb, K, p.Hp, p.Wp, p.Rp, p.Sp, p.P, p.Q};
  for (int i = 0; i < 9; ++i) inner[i] = v[i];
  return CONV_OK;
}

int conv_fwd_plan(int N, int C, int K, int H, int W, int R, int S, int dtype,
                  conv_plan_t* plan_out) {
  int st = validate_shape(N, C, K, H, W, R, S);
  if (st != CONV_OK) return st;
  if (!plan_out) return CONV_ENULL;
  if (dtype != CONV_DTYPE_F32 && dtype != CONV_DTYPE_BF16) return CONV_EINVAL;
  return cached_plan(Shape{N, C, K, H, W, R, S}, dtype, plan_out);
}

int conv_fwd_bf16_out_plan(int N, int C, int K, int H, int W, int R, int S, conv_plan_t* plan_out) {
  int st = validate_shape(N, C, K, H, W, R, S);
  if (st != CONV_OK) return st;
  if (!plan_out) return CONV_ENULL;
  Entry e;
  st = cached_entry_bf16_out(Shape{N, C, K, H, W, R, S}, ALIGN_ALL, (W - S + 1) % 8 == 0, &e);
  if (st == CONV_OK) *plan_out = e.plan;
  return st;
}

int conv_fwd_with_plan(int N, int C, int K, int H, int W, int R, int S, const void* In,
                       const void* Ker, float* Out, const conv_plan_t* plan, void* stream) {
  int st = validate_shape(N, C, K, H, W, R, S);
  if (st != CONV_OK) return st;
  if (!In || !Ker || !Out || !plan) return CONV_ENULL;
  const Shape s{N, C, K, H, W, R, S};
  conv_plan_t p = *plan;
  st = score_plan(s, &p);
  if (st != CONV_OK) return st;
  return run(s, In, Ker, Out, p, stream);
}

int conv_fwd_score_plan(int N, int C, int K, int H, int W, int R, int S, conv_plan_t* plan) {
  int st = validate_shape(N, C, K, H, W, R, S);
  if (st != CONV_OK) return st;
  if (!plan) return CONV_ENULL;
  conv_plan_t p = *plan;
  st = score_plan(Shape{N, C, K, H, W, R, S}, &p);
  if (st != CONV_OK) return st;
  *plan = p;
  return CONV_OK;
}

int conv_fwd_candidates(int N, int C, int K, int H, int W, int R, int S, int dtype,
                        conv_plan_t* plans, int cap) {
  int st = validate_shape(N, C, K, H, W, R, S);
  if (st != CONV_OK) return st;
  if (cap < 0 || (cap > 0 && !plans)) return CONV_EINVAL;
  if (dtype != CONV_DTYPE_F32 && dtype != CONV_DTYPE_BF16) return CONV_EINVAL;
  const int n = enumerate_plans(Shape{N, C, K, H, W, R, S}, dtype, plans, cap);
  return n > 0 ? n : CONV_ENOPLAN;
}

int conv_fwd_tune(int N, int C, int K, int H, int W, int R, int S, int dtype, const void* In,
                  const void* Ker, float* Out, int top_n, int reps, void* stream,
                  conv_plan_t* plan_out, float* times_us) {
  int st = validate_shape(N, C, K, H, W, R, S);
  if (st != CONV_OK) return st;
  if (!In || !Ker || !Out || !plan_out) return CONV_ENULL;
  if (dtype != CONV_DTYPE_F32 && dtype != CONV_DTYPE_BF16) return CONV_EINVAL;
  if (top_n < 1 || top_n > CONV_TUNE_MAX || reps < 1 || reps > 1000) return CONV_EINVAL;
  const Shape s{N, C, K, H, W, R, S};
  const int align = alignment_of(In, Ker);
  // the model's best plans (best first) that run with these tensors
  std::vector<conv_plan_t> buf(4096);
  const int n = enumerate_plans(s, dtype, buf.data(), (int)buf.size());
  std::vector<Entry> cand;
  for (int i = 0; i < n && i < (int)buf.size() && (int)cand.size() < top_n; ++i) {
    Entry e;
    e.plan = buf[i];
    e.v = find_variant(buf[i].variant);
    if (!e.v || !variant_fits(*e.v, dtype, align) || !resolve_geom(s, *e.v, e.plan, &e.g, nullptr)) continue;
    cand.push_back(e);
  }
  if (cand.empty()) return CONV_ENOPLAN;
  size_t best = 0;
  float best_us = 0.f;
  for (size_t i = 0; i < cand.size(); ++i) {
    float us = 0.f;
    st = time_launches(*cand[i].v, cand[i].g, In, Ker, Out, stream, reps, &us);
    if (st != CONV_OK) return st;
    if (times_us) times_us[i] = us;
    if (i == 0 || us < best_us) {
      best = i;
      best_us = us;
    }
  }
  {
    std::lock_guard<std::mutex> lk(g_mu);
    g_cache[Key{N, C, K, H, W, R, S, dtype, align}] = cand[best];
  }
  *plan_out = cand[best].plan;
  return (int)cand.size();
}

int conv_model_volume(const int perm[7], const int64_t N[7], const int64_t T[7], int out_factor,
                      double dv[3]) {
  if (!perm || !N || !T || !dv) return CONV_ENULL;
  int seen = 0;
  for (int i = 0; i < 7; ++i) {
    if (perm[i] < 0 || perm[i] > 6 || (seen >> perm[i]) & 1) return CONV_EINVAL;
    seen |= 1 << perm[i];
    if (T[i] < 1 || T[i] > N[i]) return CONV_EINVAL;
  }
  if (out_factor < 0) return CONV_EINVAL;
  model_volume(perm, N, T, out_factor, dv);
  return CONV_OK;
}

int conv_fwd_geometry(int N, int C, int K, int H, int W, int R, int S, const conv_plan_t* plan,
                      int32_t* out, int cap) {
  int st = validate_shape(N, C, K, H, W, R, S);
  if (st != CONV_OK) return st;
  if (!plan || (cap > 0 && !out)) return CONV_ENULL;
  const Variant* v = find_variant(plan->variant);
  if (!v || v->phase_skip) return CONV_EINVAL;  // phase skip: conv_fwd_ex_geometry only
  Geom g;
  int lds = 0;
  if (!resolve_geom(Shape{N, C, K, H, W, R, S}, *v, *plan, &g, &lds)) return CONV_EINVAL;
  return export_geometry(*v, g, lds, out, cap);
}

int conv_fwd_ex_geometry(int N, int C, int K, int H, int W, int R, int S, int stride_h, int stride_w, int pad_h,
                         int pad_w, const conv_plan_t* plan, int32_t* out, int cap) {
  PhaseGeom p;
  int st = phase_geom(N, C, K, H, W, R, S, stride_h, stride_w, pad_h, pad_w, &p);
  if (st != CONV_OK) return st;
  if (!plan || (cap > 0 && !out)) return CONV_ENULL;
  const Variant* v = find_variant(plan->variant);
  if (!v) return CONV_EINVAL;
  Geom g;
  int lds = 0;
  const Shape inner{N, C * p.na * p.nb, K, p.Hp, p.Wp, p.Rp, p.Sp};
  if (!resolve_geom(inner, *v, *plan, &g, &lds)) return CONV_EINVAL;
  const bool rewrite = stride_h > 1 || stride_w > 1 || pad_h > 0 || pad_w > 0;
  const bool direct = rewrite && phase_direct(*v, p, plan->dtype, &g);  // nph stays 0 where it does not apply
  if (v->phase_skip && !direct) return CONV_EINVAL;  // phase skip runs only reading In directly
  return export_geometry(*v, g, lds, out, cap);
}

int conv_fwd_release_workspaces(void* stream) { return workspace_release_stream(stream); }

const char* conv_fwd_strerror(int status) {
  switch (status) {
    case CONV_OK: return "ok";
    case CONV_EINVAL: return "invalid argument (extent <= 0, R > H, S > W, or a bad plan)";
    case CONV_ENULL: return "null pointer";
    case CONV_ERANGE: return "tensor too large (2^31 elements or more)";
    case CONV_ENOPLAN: return "no kernel configuration fits this shape";
    case CONV_EHIP: return "HIP runtime error at launch";
    case CONV_ESCRATCH: return "the call needs more scratch than the allocation-free entry point holds";
    default: return "unknown status";
  }
}

}  // extern "C"
