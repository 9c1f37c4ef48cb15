// Kernel sequences of one reversible stage (host side).
//
// Forward of a residual function Phi = conv-BN[-ReLU-conv-BN...] on input u,
// coupled as y = r + Phi(u) (Sec. 3.2):
//   conv_l (BN_{l-1}+ReLU applied in the prologue; BN partials in the epilogue)
//   -> finalize BN_l -> ... -> combine_fwd y = r + BN_L(h_L).
// Backward of the couplings in reverse order (Eq. 4-5).  For each residual
// function, given its output-side stream v, the gradient d of the coupling
// output and the residual gradient rg:
//   recompute:  the convs again (running statistics move here only, Sec. 4.1),
//               then the reconstruction x = v - BN_L(h_L);
//   gradient:   BN_L backward coefficients from partials of (d, h_L), then per
//               layer from the top an input-gradient conv whose prologue forms
//               dh_l = BN_l backward of its input on the fly and whose epilogue
//               applies the ReLU mask of the layer below and emits that layer's
//               BN-backward partials, or, for the first layer, adds rg
//               (dout = rg + dPhi/du^T d) and emits the BN_L-backward partials of
//               the next function visited; the weight gradient of each conv runs
//               on a side stream from the same on-the-fly dh (split rows,
//               fixed-order reduce into the accumulator, scaled 1/k).
// The recompute of the next function runs on its own stream while the gradient
// chain of the current one proceeds; two scratch sets alternate between them.
#include <algorithm>
#include <cstring>

#include "stage.h"

namespace petra {

namespace {

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace

Stage::Stage(const petra_stage_desc& d) : desc(d) {
  dt = d.dtype == PETRA_BF16 ? DT_BF16 : DT_FP32;
  // one backward stream: the weight gradients are deferred and grouped (with
  // three streams they run layer by layer beside the chain; measured slower
  // for every block kind)
  bwd_streams = 1;
  esz = dt == DT_BF16 ? 2 : 4;
  M = static_cast<long>(d.n) * d.h * d.w;
  const int c = d.c_half, cm = d.c_mid;

  // Canonical order: block, function F then G, conv; each conv followed by its BN.
  struct Shape { int cout, r, s, cin; };
  std::vector<Shape> fn_shapes;
  if (d.kind == PETRA_BLOCK_BASIC)
    fn_shapes = {{c, 3, 3, c}, {c, 3, 3, c}};
  else
    fn_shapes = {{cm, 1, 1, c}, {cm, 3, 3, cm}, {c, 1, 1, cm}};
  cmax = 0;
  for (auto& s : fn_shapes) cmax = std::max(cmax, std::max(s.cout, s.cin));

  // Flat layout: all conv weights first (weight-decayed range), then per BN gamma, beta.
  int64_t woff = 0;
  for (int b = 0; b < d.num_blocks; ++b)
    for (int f = 0; f < 2; ++f)
      for (auto& s : fn_shapes) woff += static_cast<int64_t>(s.cout) * s.r * s.s * s.cin;
  n_conv = woff;
  int64_t w_cur = 0, bn_cur = n_conv, run_cur = 0;
  blocks.resize(d.num_blocks);
  for (int b = 0; b < d.num_blocks; ++b) {
    for (int f = 0; f < 2; ++f) {
      ResidualFn fn{};
      fn.nconv = static_cast<int>(fn_shapes.size());
      for (size_t l = 0; l < fn_shapes.size(); ++l) {
        const Shape& s = fn_shapes[l];
        ConvLayer cv{};
        cv.cin = s.cin; cv.cout = s.cout; cv.r = s.r; cv.s = s.s; cv.pad = (s.r - 1) / 2;
        cv.w_off = w_cur;
        cv.dg_off = w_cur;  // the transposed copy uses the same offsets in its own buffer
        const int64_t numel = static_cast<int64_t>(s.cout) * s.r * s.s * s.cin;
        w_cur += numel;
        BnLayer bnl{};
        bnl.c = s.cout;
        bnl.g_off = bn_cur;
        bnl.b_off = bn_cur + s.cout;
        bnl.run_off = run_cur;
        bn_cur += 2 * s.cout;
        run_cur += s.cout;
        cv.bn = static_cast<int>(bns.size());
        bns.push_back(bnl);
        fn.conv[l] = static_cast<int>(convs.size());
        convs.push_back(cv);

        petra_param_info wi{};
        wi.offset = cv.w_off; wi.numel = numel; wi.role = PETRA_ROLE_CONV_WEIGHT; wi.ndim = 4;
        wi.shape[0] = s.cout; wi.shape[1] = s.r; wi.shape[2] = s.s; wi.shape[3] = s.cin;
        wi.weight_decay = 1; wi.bn_index = cv.bn;
        infos.push_back(wi);
        petra_param_info gi{};
        gi.offset = bnl.g_off; gi.numel = s.cout; gi.role = PETRA_ROLE_BN_GAMMA; gi.ndim = 1;
        gi.shape[0] = s.cout; gi.weight_decay = 0; gi.bn_index = cv.bn;
        infos.push_back(gi);
        petra_param_info bi = gi;
        bi.offset = bnl.b_off; bi.role = PETRA_ROLE_BN_BETA;
        infos.push_back(bi);
      }
      if (f == 0) blocks[b].f = fn; else blocks[b].g = fn;
    }
  }
  n_params = bn_cur;
  n_bnch = run_cur;
  segs.nseg = static_cast<int>(convs.size());
  for (size_t i = 0; i < convs.size() && i < static_cast<size_t>(MAX_WEIGHT_SEGS); ++i) {
    const ConvLayer& cv = convs[i];
    segs.seg[i] = WeightSeg{cv.w_off, cv.w_off, cv.dg_off, cv.cout, cv.r, cv.s, cv.cin, cv.cin};
    max_wnumel = std::max<int64_t>(max_wnumel, static_cast<int64_t>(cv.cout) * cv.r * cv.s * cv.cin);
  }

  // Workspace plan.
  int tiles_max = 1;
  for (auto& s : fn_shapes) tiles_max = std::max(tiles_max, ew_tiles(M, s.cout));
  for (const ConvLayer& cv : convs) {
    ConvArgs f = conv_args(cv);
    f.c_in = cv.cin; f.c_out = cv.cout; f.k_tot = cv.r * cv.s * cv.cin;
    ConvArgs g = conv_args(cv);
    g.c_in = cv.cout; g.c_out = cv.cin; g.k_tot = cv.r * cv.s * cv.cout;
    // the input-gradient convs run with the BN-backward prologue
    ConvArgs gb = g;
    gb.pro_h = reinterpret_cast<const void*>(16);
    for (int ep : {EP_STATS, EP_MASK, EP_RESID_STATS}) {
      tiles_max = std::max(tiles_max, conv_row_tiles(dt, f, ep));
      tiles_max = std::max(tiles_max, conv_row_tiles(dt, g, ep));
      if (ep != EP_STATS) tiles_max = std::max(tiles_max, conv_row_tiles(dt, gb, ep));
    }
  }
  // each conv layer has its own weight-gradient partials, so their reduces can
  // wait until the end of the backward and run as one launch
  int64_t wtot = 0;
  wpart_off.clear();
  for (auto& cv : convs) {
    int sp, rps;
    wgrad_splits(cv, &sp, &rps);
    wpart_off.push_back(wtot);
    wtot += (static_cast<int64_t>(sp) * cv.cout * cv.r * cv.s * cv.cin + 63) / 64 * 64;
  }
  wpart_floats = wtot;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  // deferred weight gradients: every layer on the transposed-read kernel
  {
    defer_wgrad = dt == DT_BF16 && blocks.size() >= 1;
    for (const ConvLayer& cv : convs) {
      WgradArgs w{};
      w.n = desc.n; w.h = desc.h; w.w = desc.w; w.p = desc.h; w.q = desc.w;
      w.c_in = cv.cin; w.c_out = cv.cout; w.r = cv.r; w.s = cv.s; w.stride = 1; w.pad = cv.pad;
      w.k_tot = cv.r * cv.s * cv.cin; w.m = static_cast<int>(M);
      w.dh_h = reinterpret_cast<const void*>(16);   // marks dh formed on the fly
      int sp = 0;
      if (wgrad_tr_plan(dt, w, &sp) == 0) defer_wgrad = false;
    }
  }
  couple_fwd = false;
  if (!blocks.empty() && blocks[0].f.nconv == 3) {
    const ConvLayer& cv = convs[blocks[0].f.conv[2]];
    ConvArgs a = conv_args(cv);
    a.c_in = cv.cin; a.c_out = cv.cout; a.k_tot = cv.r * cv.s * cv.cin;
    couple_fwd = conv1x1_couple_ok(dt, a);
    const ConvLayer& c0 = convs[blocks[0].g.conv[0]];
    ConvArgs b = conv_args(c0);
    b.c_in = c0.cin; b.c_out = c0.cout; b.k_tot = c0.r * c0.s * c0.cin;
    couple_next = couple_fwd && conv1x1_couple_next_ok(dt, a, b);
  }
  const int nfn = 2 * static_cast<int>(blocks.size());
  plan_b.assign(defer_wgrad ? std::max(2, nfn) : 2, ScratchPlan{});
  off_wfwd = take(static_cast<size_t>(n_conv) * esz);
  off_wdg = take(static_cast<size_t>(n_conv) * esz);
  std::vector<ScratchPlan*> plans{&plan_f};
  for (ScratchPlan& pb : plan_b) plans.push_back(&pb);
  for (ScratchPlan* p : plans) {
    for (size_t l = 0; l < 3; ++l)
      p->h[l] = l >= fn_shapes.size()                        ? 0
                : p == &plan_f && couple_fwd && l == 2       ? NO_BUF
                : take(static_cast<size_t>(M) * fn_shapes[l].cout * esz);
    const bool bwd = p != &plan_f;
    p->d1[0] = bwd ? take(static_cast<size_t>(M) * cmax * esz) : 0;
    p->d1[1] = bwd && fn_shapes.size() > 2 ? take(static_cast<size_t>(M) * cmax * esz) : 0;
    p->part = take(static_cast<size_t>(tiles_max) * 3 * cmax * sizeof(float));
    p->gpart = bwd ? take(static_cast<size_t>(tiles_max) * 2 * cmax * sizeof(float)) : 0;
    p->bpart = bwd ? take(static_cast<size_t>(tiles_max) * 2 * cmax * sizeof(float)) : 0;
    p->bnp = take(static_cast<size_t>(3) * 8 * cmax * sizeof(float));
    if (p == &plan_f) fwd_need = off;   // compute copies + the forward's scratch set
  }
  off_wpart = take(static_cast<size_t>(wpart_floats) * sizeof(float));
  if (defer_wgrad && blocks.size() > 1)
    off_inter = take(static_cast<size_t>(blocks.size() - 1) * 4 * M * desc.c_half * esz);
  ws_need = off;
}

Stage::~Stage() {
  // graph executables reference the streams and events below: release them first
  graphs.clear();
  if (ev_fork) (void)hipEventDestroy(ev_fork);
  if (ev_fwd) (void)hipEventDestroy(ev_fwd);
  if (ev_bwd) (void)hipEventDestroy(ev_bwd);
  for (hipEvent_t e : {ev_start, ev_d, ev_rec_end, ev_rec[0], ev_rec[1], ev_gdone[0],
                       ev_gdone[1], ev_wgdone[0], ev_wgdone[1]})
    if (e) (void)hipEventDestroy(e);
  if (s_wg) (void)hipStreamDestroy(s_wg);
  if (s_rec) (void)hipStreamDestroy(s_rec);
  if (s_fwd) (void)hipStreamDestroy(s_fwd);
  if (s_bwd) (void)hipStreamDestroy(s_bwd);
}

Scratch Stage::carve(const ScratchPlan& p, char* base, bool bwd) const {
  const int nl = blocks.empty() ? 0 : blocks[0].f.nconv;
  Scratch s;
  for (int l = 0; l < 3; ++l) s.h[l] = l < nl && p.h[l] != NO_BUF ? base + p.h[l] : nullptr;
  s.d1[0] = bwd ? base + p.d1[0] : nullptr;
  s.d1[1] = bwd && nl > 2 ? base + p.d1[1] : nullptr;
  s.part = reinterpret_cast<float*>(base + p.part);
  s.gpart = bwd ? reinterpret_cast<float*>(base + p.gpart) : nullptr;
  s.bpart = bwd ? reinterpret_cast<float*>(base + p.bpart) : nullptr;
  s.bnp = reinterpret_cast<float*>(base + p.bnp);
  return s;
}

void Stage::bind(float* th, float* gr, float* mo, float* rm, float* rv, void* w) {
  theta = th; grad = gr; mom = mo; rmean = rm; rvar = rv;
  ws = static_cast<char*>(w);
  sb.assign(plan_b.size(), Scratch{});
  if (ws == nullptr) {
    // bound for the scratch-free forward only: no workspace-backed pointers
    wfwd = wdg = nullptr;
    sf = Scratch{};
    wpart = nullptr;
    reset_view();
    graphs.clear();
    return;
  }
  wfwd = ws + off_wfwd;
  wdg = ws + off_wdg;
  reset_view();
  sf = carve(plan_f, ws, false);
  for (size_t i = 0; i < plan_b.size(); ++i) sb[i] = carve(plan_b[i], ws, true);
  wpart = reinterpret_cast<float*>(ws + off_wpart);
  // cached graphs hold the previous buffers' device pointers in their kernel arguments
  graphs.clear();
}

hipError_t Stage::ensure_streams() {
  if (s_fwd) return hipSuccess;
  hipError_t e;
  if ((e = hipStreamCreateWithFlags(&s_fwd, hipStreamNonBlocking)) != hipSuccess) return e;
  if ((e = hipStreamCreateWithFlags(&s_bwd, hipStreamNonBlocking)) != hipSuccess) return e;
  if ((e = hipEventCreateWithFlags(&ev_fork, hipEventDisableTiming)) != hipSuccess) return e;
  if ((e = hipEventCreateWithFlags(&ev_fwd, hipEventDisableTiming)) != hipSuccess) return e;
  if ((e = hipStreamCreateWithFlags(&s_wg, hipStreamNonBlocking)) != hipSuccess) return e;
  if ((e = hipStreamCreateWithFlags(&s_rec, hipStreamNonBlocking)) != hipSuccess) return e;
  for (hipEvent_t* ev : {&ev_start, &ev_d, &ev_rec_end, &ev_side, &ev_rec[0], &ev_rec[1], &ev_gdone[0],
                         &ev_gdone[1], &ev_wgdone[0], &ev_wgdone[1]})
    if ((e = hipEventCreateWithFlags(ev, hipEventDisableTiming)) != hipSuccess) return e;
  return hipEventCreateWithFlags(&ev_bwd, hipEventDisableTiming);
}

void Stage::sync_weights(hipStream_t st) {
  prof.begin(st);
  refresh_weights(dt, theta, segs, max_wnumel, wfwd, wdg, st);
  prof.end(K_REFRESH, st, 0.0, static_cast<double>(n_conv) * (4.0 + 2.0 * esz));
}

ConvArgs Stage::conv_args(const ConvLayer& cv) const {
  ConvArgs a{};
  a.n = desc.n; a.h = desc.h; a.w = desc.w;
  a.p = desc.h; a.q = desc.w;
  a.r = cv.r; a.s = cv.s; a.stride = 1; a.pad = cv.pad;
  a.m = static_cast<int>(M);
  return a;
}

void Stage::wgrad_splits(const ConvLayer& cv, int* splits, int* rows_per_split) const {
  WgradArgs w{};
  w.n = desc.n; w.h = desc.h; w.w = desc.w; w.p = desc.h; w.q = desc.w;
  w.c_in = cv.cin; w.c_out = cv.cout; w.r = cv.r; w.s = cv.s; w.stride = 1; w.pad = cv.pad;
  w.k_tot = cv.r * cv.s * cv.cin; w.m = static_cast<int>(M);
  w.dh_h = reinterpret_cast<const void*>(16);   // dh is always formed on the fly (marker)
  int tr_splits = 0;
  if (wgrad_tr_plan(dt, w, &tr_splits) != 0) {
    *splits = tr_splits;
    *rows_per_split = 0;
    return;
  }
  const int hshape = wgrad_halo_shape(dt, w);
  if (hshape != 0) {
    // pixel tiles strided over `splits` workgroups per (output tile, channel chunk)
    const int ntiles = wgrad_halo_tiles(dt, w);
    const int bo = hshape == 1 ? 32 : 64;
    const int per_split = ((cv.cout + bo - 1) / bo) * (cv.cin / 32);
    *splits = std::max(1, std::min(ntiles, 512 / std::max(1, per_split)));
    *rows_per_split = 0;
    return;
  }
  // About two workgroups per CU in total, each over at least 512 rows.
  const int ktot = cv.r * cv.s * cv.cin;
  const int bo = cv.cout <= 32 ? 32 : 64;
  const int tiles = ((ktot + 63) / 64) * ((cv.cout + bo - 1) / bo);
  int sp = std::max(1, 512 / std::max(1, tiles));
  long rps = (M + sp - 1) / sp;
  rps = std::max<long>(rps, 512);
  rps = (rps + 31) / 32 * 32;
  sp = static_cast<int>((M + rps - 1) / rps);
  *splits = sp;
  *rows_per_split = static_cast<int>(rps);
}

void Stage::fn_recompute(const ResidualFn& fn, const void* u, Scratch& s, bool running,
                         hipStream_t st, bool stats_only_last, bool first_done) {
  for (int l = 0; l < fn.nconv; ++l) {
    const bool stats_only = stats_only_last && l == fn.nconv - 1;
    const bool done = first_done && l == 0;
    const ConvLayer& cv = convs[fn.conv[l]];
    const BnLayer& bn = bns[cv.bn];
    ConvArgs a = conv_args(cv);
    a.src = l == 0 ? u : s.h[l - 1];
    a.c_in = cv.cin;
    a.c_split = cv.cin;
    if (l > 0) {
      a.pro_scale = s.vec(l - 1, V_SCALE, cmax);
      a.pro_shift = s.vec(l - 1, V_SHIFT, cmax);
    }
    a.wt = static_cast<const char*>(v_wf) + cv.w_off * esz;
    a.out = stats_only ? nullptr : s.h[l];
    a.c_out = cv.cout;
    a.k_tot = cv.r * cv.s * cv.cin;
    a.partials = s.part;
    if (a.out == nullptr && !(stats_only && conv1x1_couple_ok(dt, a))) {
      launch_error = true;   // no buffer for this output (not reached by the library's calls)
      return;
    }
    const int tiles = conv_row_tiles(dt, a, EP_STATS);
    if (!done) {
      prof.begin(st);
      conv(a, EP_STATS, st);
      prof.end(K_CONV_FPROP, st, 2.0 * M * cv.cout * a.k_tot,
               static_cast<double>(esz) *
                   (static_cast<double>(M) * (cv.cin + (stats_only ? 0 : cv.cout)) +
                    static_cast<double>(cv.cout) * a.k_tot));
    }
    prof.begin(st);
    bn_stats_finalize(s.part, tiles, cv.cout, M, v_th + bn.g_off, v_th + bn.b_off, desc.bn_eps,
                      s.vec(l, V_SCALE, cmax), s.vec(l, V_SHIFT, cmax), s.vec(l, V_MEAN, cmax),
                      s.vec(l, V_RSTD, cmax), running ? rmean + bn.run_off : nullptr,
                      running ? rvar + bn.run_off : nullptr, desc.bn_momentum, st);
    prof.end(K_BN_FINALIZE, st, 0.0, 8.0 * tiles * cv.cout);
  }
}

bool Stage::fn_forward(const ResidualFn& fn, const void* u, const void* r, void* y, Scratch& s,
                       hipStream_t st, bool first_done, const ResidualFn* next) {
  // with couple_fwd the last conv writes its statistics only
  fn_recompute(fn, u, s, false, st, couple_fwd, first_done);
  // y = r + BN_L(h_L), and (couple_next) the next function's first conv on y,
  // into the same scratch set
  return coupling(fn, s, r, y, false, st, next, &s);
}

bool Stage::coupling(const ResidualFn& fn, Scratch& s, const void* r, void* out, bool sub,
                     hipStream_t st, const ResidualFn* next, Scratch* ns) {
  const int L = fn.nconv - 1;
  const ConvLayer& cv = convs[fn.conv[L]];
  const int c = cv.cout;
  if (couple_next && next != nullptr && ns != nullptr) {
    const ConvLayer& c0 = convs[next->conv[0]];
    ConvArgs a = conv_args(cv);
    a.src = s.h[L - 1];
    a.c_in = cv.cin;
    a.c_split = cv.cin;
    a.pro_scale = s.vec(L - 1, V_SCALE, cmax);
    a.pro_shift = s.vec(L - 1, V_SHIFT, cmax);
    a.wt = static_cast<const char*>(v_wf) + cv.w_off * esz;
    a.out = out;
    a.resid = r;
    a.c_out = c;
    a.k_tot = cv.r * cv.s * cv.cin;
    const NextConv nx{static_cast<const char*>(v_wf) + c0.w_off * esz, ns->h[0], ns->part};
    prof.begin(st);
    if (!conv1x1_couple(dt, a, s.vec(L, V_SCALE, cmax), s.vec(L, V_SHIFT, cmax), sub, st, &nx))
      launch_error = true;
    prof.end(K_CONV_FPROP, st, 2.0 * M * (c * a.k_tot + c0.cout * c0.cin),
             static_cast<double>(esz) *
                 (static_cast<double>(M) * (cv.cin + 2.0 * c + c0.cout) +
                  static_cast<double>(c) * a.k_tot + static_cast<double>(c0.cout) * c0.cin));
    return true;
  }
  if (couple_fwd) {
    // h_L recomputed from the layer's input (the same bits as the statistics pass)
    ConvArgs a = conv_args(cv);
    a.src = s.h[L - 1];
    a.c_in = cv.cin;
    a.c_split = cv.cin;
    a.pro_scale = s.vec(L - 1, V_SCALE, cmax);
    a.pro_shift = s.vec(L - 1, V_SHIFT, cmax);
    a.wt = static_cast<const char*>(v_wf) + cv.w_off * esz;
    a.out = out;
    a.resid = r;
    a.c_out = c;
    a.k_tot = cv.r * cv.s * cv.cin;
    prof.begin(st);
    if (!conv1x1_couple(dt, a, s.vec(L, V_SCALE, cmax), s.vec(L, V_SHIFT, cmax), sub, st))
      launch_error = true;
    prof.end(K_CONV_FPROP, st, 2.0 * M * c * a.k_tot,
             static_cast<double>(esz) * (static_cast<double>(M) * (cv.cin + 2.0 * c) +
                                         static_cast<double>(c) * a.k_tot));
    return false;
  }
  prof.begin(st);
  if (sub)
    combine_rec(dt, r, s.h[L], s.vec(L, V_SCALE, cmax), s.vec(L, V_SHIFT, cmax), out, M, c, st);
  else
    combine_fwd(dt, r, s.h[L], s.vec(L, V_SCALE, cmax), s.vec(L, V_SHIFT, cmax), out, M, c, st);
  prof.end(sub ? K_COMBINE_BWD : K_COMBINE_FWD, st, 0.0, 3.0 * M * c * esz);
  return false;
}

bool Stage::conv(const ConvArgs& a, int ep, hipStream_t st) {
  const bool ok = conv_gemm(dt, a, ep, st);
  if (!ok) launch_error = true;
  return ok;
}

// Gradient chain of one residual function (enqueue only), in two parts so the
// recompute of the next function can be enqueued between them: part 0 is the
// BN_L-backward coefficients and the layers L..1, part 1 the first layer.  s
// holds the function's recomputed h and BN statistics and, in gpart, the
// BN_L-backward partials of its output gradient d.  next/sn: the function
// visited next (recompute enqueued before part 1), whose BN_L-backward partials
// the first-layer conv emits.  Each layer's input-gradient conv is enqueued
// before its weight gradient, which runs on the side stream.
void Stage::fn_grad(const BwdFn& f, Scratch& s, const BwdFn* next, Scratch* sn, hipStream_t st,
                    hipStream_t wst, hipStream_t rs, bool wait_prev_wg, int parity, int part,
                    const void** dsrc_io) {
  const ResidualFn& fn = *f.fn;
  const bool wb = wst != st;  // weight gradients on their own stream
  const bool rb = rs != st;   // recompute on its own stream
  const float inv_k = 1.0f / static_cast<float>(std::max(1, opt.accum_k));
  const int L = fn.nconv - 1;
  if (part == 0) {
    const ConvLayer& cv = convs[fn.conv[L]];
    const BnLayer& bn = bns[cv.bn];
    prof.begin(st);
    bn_bwd_finalize(s.gpart, s.gtiles, cv.cout, M, v_th + bn.g_off, s.vec(L, V_MEAN, cmax),
                    s.vec(L, V_RSTD, cmax), inv_k, grad + bn.g_off, grad + bn.b_off,
                    s.vec(L, V_CA, cmax), s.vec(L, V_CB, cmax), s.vec(L, V_CC, cmax), st);
    prof.end(K_BN_BWD_FINALIZE, st, 0.0, 8.0 * s.gtiles * cv.cout);
    *dsrc_io = f.d;
  }
  const int l_hi = part == 0 ? L : 0, l_lo = part == 0 ? 1 : 0;
  for (int l = l_hi; l >= l_lo; --l) {
    const ConvLayer& cv = convs[fn.conv[l]];
    const void* dsrc = *dsrc_io;
    // Both consumers form dh_l = BN_l backward of dsrc on the fly from (dsrc, h_l).
    if (wb) PETRA_HIP(hip_status, hipEventRecord(ev_d, st));
    // input gradient: conv of dh_l with the transposed, flipped weights
    ConvArgs a = conv_args(cv);
    a.src = dsrc;
    a.c_in = cv.cout;
    a.c_split = cv.cout;
    a.pro_h = s.h[l];
    a.pro_ca = s.vec(l, V_CA, cmax);
    a.pro_cb = s.vec(l, V_CB, cmax);
    a.pro_cc = s.vec(l, V_CC, cmax);
    a.pro_mean = s.vec(l, V_MEAN, cmax);
    a.wt = static_cast<const char*>(v_wd) + cv.dg_off * esz;
    a.c_out = cv.cin;
    a.k_tot = cv.r * cv.s * cv.cout;
    const double dbytes = static_cast<double>(esz) *
                          (static_cast<double>(M) * (2.0 * cv.cout + 2.0 * cv.cin) +
                           static_cast<double>(cv.cin) * a.k_tot);
    if (l > 0) {
      const ConvLayer& lo = convs[fn.conv[l - 1]];
      const BnLayer& bl = bns[lo.bn];
      a.out = s.d1[(L - l) & 1];
      a.ep_h = s.h[l - 1];
      a.ep_scale = s.vec(l - 1, V_SCALE, cmax);
      a.ep_shift = s.vec(l - 1, V_SHIFT, cmax);
      a.ep_mean = s.vec(l - 1, V_MEAN, cmax);
      a.ep_rstd = s.vec(l - 1, V_RSTD, cmax);
      a.partials = s.bpart;
      const int tiles_conv = conv_row_tiles(dt, a, EP_MASK);
      prof.begin(st);
      conv(a, EP_MASK, st);
      prof.end(K_CONV_DGRAD, st, 2.0 * M * cv.cin * a.k_tot, dbytes);
      prof.begin(st);
      bn_bwd_finalize(s.bpart, tiles_conv, lo.cout, M, v_th + bl.g_off, s.vec(l - 1, V_MEAN, cmax),
                      s.vec(l - 1, V_RSTD, cmax), inv_k, grad + bl.g_off, grad + bl.b_off,
                      s.vec(l - 1, V_CA, cmax), s.vec(l - 1, V_CB, cmax),
                      s.vec(l - 1, V_CC, cmax), st);
      prof.end(K_BN_BWD_FINALIZE, st, 0.0, 8.0 * tiles_conv * lo.cout);
      *dsrc_io = s.d1[(L - l) & 1];
    } else {
      a.out = f.dout;
      a.resid = f.rg;
      // dout may alias the previous function's output gradient, which that
      // function's weight gradients read
      if (wb && wait_prev_wg) PETRA_HIP(hip_status, hipStreamWaitEvent(st, ev_wgdone[parity ^ 1], 0));
      if (next != nullptr) {
        if (rb) PETRA_HIP(hip_status, hipStreamWaitEvent(st, ev_rec[parity ^ 1], 0));
        const int NL = next->fn->nconv - 1;
        a.ep_h = sn->h[NL];
        a.ep_mean = sn->vec(NL, V_MEAN, cmax);
        a.ep_rstd = sn->vec(NL, V_RSTD, cmax);
        a.partials = sn->gpart;
        sn->gtiles = conv_row_tiles(dt, a, EP_RESID_STATS);
        prof.begin(st);
        conv(a, EP_RESID_STATS, st);
        prof.end(K_CONV_DGRAD, st, 2.0 * M * cv.cin * a.k_tot, dbytes + 2.0 * esz * M * cv.cin);
      } else {
        prof.begin(st);
        conv(a, EP_RESID, st);
        prof.end(K_CONV_DGRAD, st, 2.0 * M * cv.cin * a.k_tot, dbytes);
      }
    }
    // weight gradient of conv_l (side stream), from the same dsrc and h_l
    if (wb) PETRA_HIP(hip_status, hipStreamWaitEvent(wst, ev_d, 0));
    WgradArgs w{};
    w.dh = dsrc;
    w.dh_h = s.h[l];
    w.dh_ca = s.vec(l, V_CA, cmax);
    w.dh_cb = s.vec(l, V_CB, cmax);
    w.dh_cc = s.vec(l, V_CC, cmax);
    w.dh_mean = s.vec(l, V_MEAN, cmax);
    w.src = l == 0 ? f.u : s.h[l - 1];
    w.c_split = cv.cin;
    if (l > 0) {
      w.pro_scale = s.vec(l - 1, V_SCALE, cmax);
      w.pro_shift = s.vec(l - 1, V_SHIFT, cmax);
    }
    const int64_t poff = wpart_off[static_cast<size_t>(&cv - convs.data())];
    w.partials = wpart + poff;
    w.n = desc.n; w.h = desc.h; w.w = desc.w; w.c_in = cv.cin; w.p = desc.h; w.q = desc.w;
    w.c_out = cv.cout; w.r = cv.r; w.s = cv.s; w.stride = 1; w.pad = cv.pad;
    w.k_tot = cv.r * cv.s * cv.cin;
    w.m = static_cast<int>(M);
    wgrad_splits(cv, &w.splits, &w.rows_per_split);
    const double wnumel = static_cast<double>(cv.cout) * w.k_tot;
    TrSeg seg{};
    if (defer_cur) {
      // launched with the other deferred layers at the end of the backward
      (void)wgrad_tr_segment(dt, w, static_cast<long>(poff), static_cast<long>(cv.w_off), &seg);
      pending_wgrad.push_back(w);
      pending_reduce.push_back(seg);
      continue;
    }
    prof.begin(wst);
    conv_wgrad(dt, w, wst);
    prof.end(K_CONV_WGRAD, wst, 2.0 * M * wnumel,
             static_cast<double>(esz) * M * (cv.cin + 2.0 * cv.cout) + 4.0 * w.splits * wnumel);
    if (wgrad_tr_segment(dt, w, static_cast<long>(poff), static_cast<long>(cv.w_off), &seg)) {
      pending_reduce.push_back(seg);   // reduced at the end of the backward
    } else {
      prof.begin(wst);
      wgrad_reduce(w.partials, w.splits, static_cast<long>(cv.cout) * w.k_tot, inv_k,
                   grad + cv.w_off, wst);
      prof.end(K_WGRAD_REDUCE, wst, 0.0, 4.0 * wnumel * (w.splits + 2));
    }
  }
  if (part == 1) {
    if (rb) PETRA_HIP(hip_status, hipEventRecord(ev_gdone[parity], st));
    if (wb || rs != wst) PETRA_HIP(hip_status, hipEventRecord(ev_wgdone[parity], wst));
  }
}

void Stage::forward(const void* x1, const void* x2, void* y1, void* y2, hipStream_t st) {
  forward_with(x1, x2, y1, y2, sf, st);
}

void Stage::forward_on(char* base, const void* x1, const void* x2, void* y1, void* y2,
                       hipStream_t st) {
  void* wf = base + off_wfwd;
  void* wd = base + off_wdg;
  // the compute copies of the current master parameters, then the forward
  refresh_weights(dt, theta, segs, max_wnumel, wf, wd, st);
  Scratch s = carve(plan_f, base, false);
  const float* th0 = v_th;
  const void* wf0 = v_wf;
  const void* wd0 = v_wd;
  const bool pe = prof.enabled;
  prof.enabled = false;   // no timing events (they would be created on first use)
  set_view(theta, wf, wd);
  forward_with(x1, x2, y1, y2, s, st);
  set_view(th0, wf0, wd0);
  prof.enabled = pe;
}

void Stage::forward_with(const void* x1, const void* x2, void* y1, void* y2, Scratch& s,
                         hipStream_t st) {
  const void* a1 = x1;
  const void* a2 = x2;
  bool done = false;   // the next function's first conv ran inside a coupling
  for (size_t bi = 0; bi < blocks.size(); ++bi) {
    const Block& b = blocks[bi];
    const ResidualFn* after = bi + 1 < blocks.size() ? &blocks[bi + 1].f : nullptr;
    done = fn_forward(b.f, a2, a1, y1, s, st, done, &b.g);    // y1 = x1 + F(x2)
    done = fn_forward(b.g, y1, a2, y2, s, st, done, after);   // y2 = x2 + G(y1)
    a1 = y1;
    a2 = y2;
  }
}

void Stage::reconstruct(const void* y1, const void* y2, void* x1, void* x2, hipStream_t st) {
  Scratch& s = sb[0];
  const void* c1 = y1;
  const void* c2 = y2;
  for (int b = static_cast<int>(blocks.size()) - 1; b >= 0; --b) {
    const Block& blk = blocks[b];
    // x2 = y2 - G(y1), then x1 = y1 - F(x2); in place across blocks
    for (int f = 0; f < 2; ++f) {
      const ResidualFn& fn = f == 0 ? blk.g : blk.f;
      const void* u = f == 0 ? c1 : x2;
      const void* v = f == 0 ? c2 : c1;
      void* out = f == 0 ? x2 : x1;
      fn_recompute(fn, u, s, false, st);
      coupling(fn, s, v, out, true, st);
    }
    c1 = x1;
    c2 = x2;
  }
}

void Stage::backward(const void* y1, const void* y2, const void* dy1, const void* dy2, void* x1,
                     void* x2, void* dx1, void* dx2, hipStream_t st, hipStream_t side) {
  // Residual functions in the order the backward visits them.
  pending_reduce.clear();
  pending_wgrad.clear();
  // streams: the weight gradients (2+) and the recompute of the next function
  // (3) on side streams; one stream when profiling per launch
  const bool par = s_rec != nullptr && s_wg != nullptr && !prof.enabled;
  hipStream_t rs = par && bwd_streams >= 3 ? s_rec : st;
  hipStream_t wst = par && bwd_streams >= 2 ? s_wg : st;
  const bool rb = rs != st, wb = wst != st;
  // single stream: the weight gradients wait for the end (the first function's
  // only when its inputs survive the backward)
  const bool defer = defer_wgrad && !rb && !wb;
  std::vector<BwdFn> fl;
  const void* c1 = y1;
  const void* c2 = y2;
  const void* g1 = dy1;
  const void* g2 = dy2;
  const size_t half = static_cast<size_t>(M) * desc.c_half * esz;
  for (int b = static_cast<int>(blocks.size()) - 1; b >= 0; --b) {
    const Block& blk = blocks[b];
    // blocks 1.. write to their own buffers when the weight gradients are deferred
    char* ib = defer && b > 0 ? ws + off_inter + static_cast<size_t>(b - 1) * 4 * half : nullptr;
    void* bx1 = ib ? ib : x1;
    void* bx2 = ib ? ib + half : x2;
    void* bdx1 = ib ? ib + 2 * half : dx1;
    void* bdx2 = ib ? ib + 3 * half : dx2;
    // x2 = y2 - G(y1); z1 = g1 + dG/dy1^T g2  (written to dx1)
    fl.push_back(BwdFn{&blk.g, c1, c2, g2, g1, bx2, bdx1});
    // x1 = y1 - F(x2); dx2 = g2 + dF/dx2^T z1
    fl.push_back(BwdFn{&blk.f, bx2, c1, bdx1, g2, bx1, bdx2});
    c1 = bx1; c2 = bx2; g1 = bdx1; g2 = bdx2;
  }
  const int nf = static_cast<int>(fl.size());
  std::vector<char> first_done(static_cast<size_t>(nf), 0);   // first conv run by a coupling
  // scratch set of function f: its own when deferring, else alternating
  auto S = [&](int f) -> Scratch& { return defer ? sb[f] : sb[f & 1]; };
  if (rb || wb) PETRA_HIP(hip_status, hipEventRecord(ev_start, st));
  if (rb) PETRA_HIP(hip_status, hipStreamWaitEvent(rs, ev_start, 0));
  if (wb) PETRA_HIP(hip_status, hipStreamWaitEvent(wst, ev_start, 0));
  auto last_c = [&](const BwdFn& f) { return convs[f.fn->conv[f.fn->nconv - 1]].cout; };
  // First function: recompute, reconstruction and the BN_L-backward partials of
  // the given output gradient.
  {
    Scratch& s0 = S(0);
    fn_recompute(*fl[0].fn, fl[0].u, s0, true, rs);
    const int L = fl[0].fn->nconv - 1;
    const int c = last_c(fl[0]);
    prof.begin(rs);
    combine_bwd(dt, fl[0].v, s0.h[L], fl[0].d, s0.vec(L, V_SCALE, cmax),
                s0.vec(L, V_SHIFT, cmax), s0.vec(L, V_MEAN, cmax),
                s0.vec(L, V_RSTD, cmax), fl[0].xrec, s0.gpart, M, c, rs);
    prof.end(K_COMBINE_BWD, rs, 0.0, 4.0 * M * c * esz);
    s0.gtiles = ew_tiles(M, c);
    if (rb) PETRA_HIP(hip_status, hipEventRecord(ev_rec[0], rs));
  }
  for (int f = 0; f < nf; ++f) {
    const int p = f & 1;
    const bool has_next = f + 1 < nf;
    const BwdFn* nx = has_next ? &fl[f + 1] : nullptr;
    Scratch& sc = S(f);
    Scratch* sn = has_next ? &S(f + 1) : nullptr;
    const void* dsrc = nullptr;
    // the first function's weight gradients read y1 and dy2, which the last
    // function overwrites when the caller runs in place (x1 == y1, dx2 == dy2)
    defer_cur = defer && (f >= 1 || (x1 != y1 && dx2 != dy2));
    if (rb) PETRA_HIP(hip_status, hipStreamWaitEvent(st, ev_rec[p], 0));
    fn_grad(fl[f], sc, nx, sn, st, wst, rs, f >= 1, p, 0, &dsrc);
    if (has_next) {
      // recompute of the next function (its input is this function's
      // reconstruction); its scratch set was last used by function f - 1
      if (rb && f >= 1) PETRA_HIP(hip_status, hipStreamWaitEvent(rs, ev_gdone[p ^ 1], 0));
      fn_recompute(*fl[f + 1].fn, fl[f + 1].u, *sn, true, rs, false, first_done[f + 1] != 0);
      if (rb) PETRA_HIP(hip_status, hipEventRecord(ev_rec[p ^ 1], rs));
    }
    fn_grad(fl[f], sc, nx, sn, st, wst, rs, f >= 1, p, 1, &dsrc);
    if (defer && side != nullptr && ev_side != nullptr && nf >= 2 &&
        (f + 1 == nf / 2 || f + 1 == nf - 1)) {
      // the weight gradients collected so far on the idle side stream (after
      // the first half and before the last function: one event each)
      PETRA_HIP(hip_status, hipEventRecord(ev_side, st));
      PETRA_HIP(hip_status, hipStreamWaitEvent(side, ev_side, 0));
      flush_deferred(side);
    }
    if (has_next) {
      // reconstruction of the next function; it may overwrite this function's
      // input, which this function's weight gradients read
      if (rs != wst) PETRA_HIP(hip_status, hipStreamWaitEvent(rs, ev_wgdone[p], 0));
      const BwdFn& nx = fl[f + 1];
      // with one scratch set per function (one stream), the reconstruction also
      // runs the first conv of the function after next, whose input it is
      const bool fuse = defer && !rb && f + 2 < nf && fl[f + 2].u == nx.xrec;
      const bool ran = coupling(*nx.fn, *sn, nx.v, nx.xrec, true, rs,
                                fuse ? fl[f + 2].fn : nullptr, fuse ? &S(f + 2) : nullptr);
      if (fuse && ran) first_done[f + 2] = 1;
    }
  }
  defer_cur = false;
  // join the side streams
  if (rb) {
    PETRA_HIP(hip_status, hipEventRecord(ev_rec_end, rs));
    PETRA_HIP(hip_status, hipStreamWaitEvent(st, ev_rec_end, 0));
  }
  if (wb) PETRA_HIP(hip_status, hipStreamWaitEvent(st, ev_wgdone[(nf - 1) & 1], 0));
  // the (remaining) deferred weight gradients and every layer's reduce: their
  // inputs are still intact (each function kept its scratch set and its block's
  // buffers)
  flush_deferred(st);
}

void Stage::flush_deferred(hipStream_t st) {
  if (!pending_wgrad.empty()) {
    // one launch per kernel configuration (and per MAX_WG_GROUP layers)
    std::vector<std::pair<int, WgradArgs>> byplan;
    for (const WgradArgs& w : pending_wgrad) {
      int sp = 0;
      byplan.emplace_back(wgrad_tr_plan(dt, w, &sp), w);
    }
    std::stable_sort(byplan.begin(), byplan.end(),
                     [](const auto& a, const auto& b) { return a.first < b.first; });
    for (size_t i0 = 0; i0 < byplan.size();) {
      size_t i1 = i0;
      std::vector<WgradArgs> grp;
      double fl = 0.0, by = 0.0;
      while (i1 < byplan.size() && byplan[i1].first == byplan[i0].first &&
             grp.size() < static_cast<size_t>(MAX_WG_GROUP)) {
        const WgradArgs& w = byplan[i1].second;
        const double wn = static_cast<double>(w.c_out) * w.k_tot;
        fl += 2.0 * M * wn;
        by += static_cast<double>(esz) * M * (w.c_in + 2.0 * w.c_out) + 4.0 * w.splits * wn;
        grp.push_back(w);
        ++i1;
      }
      prof.begin(st);
      const bool ok = conv_wgrad_tr_group(dt, grp.data(), static_cast<int>(grp.size()), st);
      prof.end(K_CONV_WGRAD, st, fl, by);
      if (!ok) launch_error = true;
      i0 = i1;
    }
    pending_wgrad.clear();
  }
  // the deferred weight-gradient reduces of every layer, in one launch
  if (!pending_reduce.empty()) {
    const float inv_k = 1.0f / static_cast<float>(std::max(1, opt.accum_k));
    for (size_t i0 = 0; i0 < pending_reduce.size(); i0 += MAX_TR_SEGS) {
      const int n = static_cast<int>(std::min<size_t>(MAX_TR_SEGS, pending_reduce.size() - i0));
      double bytes = 0.0;
      for (int i = 0; i < n; ++i)
        bytes += 4.0 * pending_reduce[i0 + i].numel * (pending_reduce[i0 + i].splits + 2);
      prof.begin(st);
      wgrad_tr_reduce_group(wpart, pending_reduce.data() + i0, n, inv_k, grad, st);
      prof.end(K_WGRAD_REDUCE, st, 0.0, bytes);
    }
    pending_reduce.clear();
  }
}

bool Stage::update_due() const {
  const int k = std::max(1, opt.accum_k);
  return !(bwd_count == 0 || bwd_count == last_update || bwd_count % k != 0);
}

void Stage::update_kernels(hipStream_t st) {
  prof.begin(st);
  sgd_update(theta, grad, mom, n_params, n_conv, opt.lr, opt.momentum, opt.weight_decay,
             opt.nesterov, st);
  prof.end(K_SGD, st, 0.0, 24.0 * n_params);
  sync_weights(st);
}

}  // namespace petra
