// Kernel sequences and buffers of the one-GPU multi-stage schedule.
//
// Buffers per stage j (all in the caller's workspace):
//  * input ring: the front layer's input of the last 2(J - j) + 1 micro-batches
//    (stage 0: the images, padded to 8 channels; the labels ride along in a
//    ring of J).  It serves the front layer's recompute on the backward and,
//    for stage j - 1, as the reconstructed output it receives from stage j.
//    Stage j - 1's forward writes its output straight into slot m of it.
//  * gradient messages to stage j - 1, double-buffered by tick parity.
//  * front-layer scratch for the forward and for the backward, the block
//    program's own workspace, and the head's buffers in the last stage.
#include <algorithm>

#include "net.h"

namespace petra {

namespace {

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace

Net::Net(const petra_net_desc& d) : desc(d) {
  dt = d.dtype == PETRA_BF16 ? DT_BF16 : DT_FP32;
  esz = dt == DT_BF16 ? 2 : 4;
  // stage list: one per level, or the per-layer split
  struct Spec { int level; bool front; int nblocks; };
  std::vector<Spec> specs;
  for (int l = 0; l < d.num_stages; ++l) {
    if (!d.split_stages) {
      specs.push_back({l, true, d.blocks_per_stage});
      continue;
    }
    specs.push_back({l, true, 0});
    for (int b = 0; b < d.blocks_per_stage; ++b) specs.push_back({l, false, 1});
  }
  J = static_cast<int>(specs.size());
  st.resize(J);
  const int k = d.classes;
  int64_t off = 0, run = 0;
  int nfront = 0;
  for (int j = 0; j < J; ++j) {
    NetStage& s = st[j];
    const Spec& sp = specs[j];
    s.j = j;
    s.level = sp.level;
    s.has_front = sp.front;
    s.has_blocks = sp.nblocks > 0;
    s.first = j == 0;
    s.last = j == J - 1;
    const int l = sp.level;
    s.C = d.widths[l];
    s.H = d.h >> l;
    s.W = d.w >> l;
    if (s.has_front && l == 0) {
      s.Hin = d.h; s.Win = d.w; s.Cin = 8; s.cin_real = d.c_img; s.R = 3; s.stride = 1; s.pad = 1;
    } else if (s.has_front) {
      s.Hin = d.h >> (l - 1); s.Win = d.w >> (l - 1); s.Cin = d.widths[l - 1];
      s.cin_real = s.Cin; s.R = 1; s.stride = 2; s.pad = 0;
    } else {
      s.Hin = s.H; s.Win = s.W; s.Cin = s.C; s.cin_real = s.C; s.R = 0; s.stride = 1; s.pad = 0;
    }
    if (s.has_front) s.fseg = nfront++;
    s.M = static_cast<long>(d.n) * s.H * s.W;
    s.Min = static_cast<long>(d.n) * s.Hin * s.Win;
    if (s.has_blocks) {
      petra_stage_desc sd{};
      sd.n = d.n; sd.h = s.H; sd.w = s.W; sd.c_half = s.C / 2; sd.c_mid = 0;
      sd.num_blocks = sp.nblocks; sd.kind = PETRA_BLOCK_BASIC; sd.dtype = d.dtype;
      sd.bn_eps = d.bn_eps; sd.bn_momentum = d.bn_momentum;
      s.blocks.reset(new Stage(sd));
    }
    const int64_t blk_params = s.has_blocks ? s.blocks->n_params : 0;
    const int64_t blk_bnch = s.has_blocks ? s.blocks->n_bnch : 0;
    const int cf = s.has_front ? s.C : 0;
    // flat layout: [front w][fc w] (decayed) [blocks] [front gamma][front beta][fc b]
    s.off_front_w = off;
    s.n_front_w = s.has_front ? static_cast<int64_t>(s.C) * s.R * s.R * s.cin_real : 0;
    off += s.n_front_w;
    s.off_fc_w = off;
    s.n_fc_w = s.last ? static_cast<int64_t>(k) * s.C : 0;
    off += s.n_fc_w;
    s.off_decay = s.off_front_w;
    s.n_decay = s.n_front_w + s.n_fc_w;
    s.off_blocks = off;
    off += blk_params;
    s.off_front_g = off;
    s.off_front_b = off + cf;
    off += 2 * cf;
    s.off_fc_b = off;
    off += s.last ? k : 0;
    s.off_plain = s.off_front_g;
    s.n_plain = off - s.off_front_g;
    s.n_span = off - s.off_front_w;
    s.run_front = run;
    run += cf;
    s.run_blocks = run;
    run += blk_bnch;

    // canonical parameter order
    if (s.has_front) {
      petra_param_info wi{};
      wi.offset = s.off_front_w; wi.numel = s.n_front_w; wi.role = PETRA_ROLE_CONV_WEIGHT;
      wi.ndim = 4; wi.shape[0] = s.C; wi.shape[1] = s.R; wi.shape[2] = s.R; wi.shape[3] = s.cin_real;
      wi.weight_decay = 1; wi.bn_index = -1;
      infos.push_back(wi);
      petra_param_info gi{};
      gi.offset = s.off_front_g; gi.numel = s.C; gi.role = PETRA_ROLE_BN_GAMMA; gi.ndim = 1;
      gi.shape[0] = s.C; gi.weight_decay = 0; gi.bn_index = -1;
      infos.push_back(gi);
      petra_param_info bi = gi;
      bi.offset = s.off_front_b; bi.role = PETRA_ROLE_BN_BETA;
      infos.push_back(bi);
    }
    if (s.has_blocks) {
      for (petra_param_info p : s.blocks->infos) {
        p.offset += s.off_blocks;
        p.bn_index = -1;
        infos.push_back(p);
      }
    }
    if (s.last) {
      petra_param_info fw{};
      fw.offset = s.off_fc_w; fw.numel = s.n_fc_w; fw.role = PETRA_ROLE_FC_WEIGHT; fw.ndim = 2;
      fw.shape[0] = k; fw.shape[1] = s.C; fw.weight_decay = 1; fw.bn_index = -1;
      infos.push_back(fw);
      petra_param_info fb{};
      fb.offset = s.off_fc_b; fb.numel = k; fb.role = PETRA_ROLE_FC_BIAS; fb.ndim = 1;
      fb.shape[0] = k; fb.weight_decay = 0; fb.bn_index = -1;
      infos.push_back(fb);
    }
  }
  n_params = off;
  n_bnch = run;

  // front weight copies
  int64_t fw_off = 0, dg_off = 0;
  front_segs.nseg = nfront;
  for (NetStage& s : st) {
    if (!s.has_front) continue;
    front_segs.seg[s.fseg] = WeightSeg{s.off_front_w, fw_off, dg_off, s.C, s.R, s.R, s.cin_real, s.Cin};
    const int64_t padded = static_cast<int64_t>(s.C) * s.R * s.R * s.Cin;
    front_max_numel = std::max(front_max_numel, padded);
    fw_off += padded;
    dg_off += s.n_front_w;
  }

  bwd_mode = (d.input_buffer ? 1 : 0) | (d.param_buffer ? 2 : 0);
  // workspace plan
  // (each allocation is also counted, by purpose, in the stage's mem[])
  size_t o = 0;
  int64_t* cur = nullptr;
  auto take = [&](size_t bytes) {
    const size_t r = o;
    o = align_up(o + bytes, 256);
    if (cur) *cur += static_cast<int64_t>(o - r);
    return r;
  };
  o_front_wfwd = take(static_cast<size_t>(fw_off) * esz);
  o_front_wdg = take(static_cast<size_t>(dg_off) * esz);
  for (int j = 0; j < J; ++j) {
    NetStage& s = st[j];
    const size_t act = static_cast<size_t>(s.M) * s.C * esz;   // full-width block activation
    const size_t half = act / 2;
    const size_t bconv = s.has_blocks ? align_up(static_cast<size_t>(s.blocks->n_conv) * esz, 256) : 0;
    const size_t fpad = s.has_front ? static_cast<size_t>(s.C) * s.R * s.R * s.Cin : 0;
    s.mem[MEM_WEIGHT_COPIES] += static_cast<int64_t>((fpad + s.n_front_w) * esz + 2 * bconv);
    s.mem[MEM_SCRATCH] -= static_cast<int64_t>(2 * bconv);
    cur = &s.mem[MEM_SCRATCH];
    if (s.has_blocks) s.o_blocks_ws = take(s.blocks->ws_need);
    if (s.has_front) {
      s.ring_depth = s.first ? 2 * J - 1 : 2 * (J - j) + 1;
      s.ring_slot_bytes = align_up(static_cast<size_t>(s.Min) * s.Cin * esz, 256);
      cur = &s.mem[MEM_ACTIVATION_BUFFER];
      s.o_ring = take(s.ring_slot_bytes * (s.ring_depth + 1));   // + the backprop pass's slot
      s.mem[MEM_ACTIVATION_BUFFER] -= static_cast<int64_t>(s.ring_slot_bytes);
      s.mem[MEM_SCRATCH] += static_cast<int64_t>(s.ring_slot_bytes);
      cur = &s.mem[MEM_SCRATCH];
    } else {
      for (int p = 0; p < 2; ++p)
        for (int h = 0; h < 2; ++h) s.o_fin[p][h] = take(half);
      s.o_bpin = take(act);
    }
    if (!s.last && (d.input_buffer || d.param_buffer)) {
      // micro-batch m is kept from its forward (tick m + j) to its backward
      // (tick m + 2J - 2 - j)
      s.buf_depth = 2 * (J - 1 - j) + 1;
      if (d.input_buffer && s.has_blocks) {
        s.ib_slot_bytes = align_up(act, 256);
        cur = &s.mem[MEM_INPUT_BUFFER];
        s.o_ib = take(s.ib_slot_bytes * s.buf_depth);
        cur = &s.mem[MEM_SCRATCH];
      }
      if (d.param_buffer) {
        size_t q = align_up(static_cast<size_t>(s.n_span) * sizeof(float), 256);
        s.ps_bwf = q;
        q += bconv;
        s.ps_bwd = q;
        q += bconv;
        s.ps_fwf = q;
        q += align_up(fpad * esz, 256);
        s.ps_fwd = q;
        q += align_up(static_cast<size_t>(s.n_front_w) * esz, 256);
        s.ps_slot_bytes = q;
        cur = &s.mem[MEM_PARAM_BUFFER];
        s.o_ps = take(s.ps_slot_bytes * s.buf_depth);
        cur = &s.mem[MEM_SCRATCH];
      }
      if (s.has_blocks) {
        s.o_rx1 = take(half);
        s.o_rx2 = take(half);
        s.o_ry1 = take(half);
        s.o_ry2 = take(half);
      }
    }
    if (s.has_front) {
    // conv args of the front layer, for tile counts and weight-gradient splits
    ConvArgs f{};
    f.n = d.n; f.h = s.Hin; f.w = s.Win; f.c_in = s.Cin; f.p = s.H; f.q = s.W; f.c_out = s.C;
    f.r = s.R; f.s = s.R; f.stride = s.stride; f.pad = s.pad; f.k_tot = s.R * s.R * s.Cin;
    f.m = static_cast<int>(s.M);
    f.c_split = s.first ? s.Cin : s.Cin / 2;
    f.src2 = s.first ? nullptr : reinterpret_cast<const void*>(16);  // marks the two-tensor input
    const int tiles = std::max(std::max(conv_row_tiles(dt, f, EP_STATS), split_tiles(s.M, s.C)), 1);
    const size_t part = static_cast<size_t>(tiles) * 3 * s.C * sizeof(float);
    const size_t bnp = static_cast<size_t>(8) * s.C * sizeof(float);
    s.o_fh = take(act);
    s.o_fx1 = take(half);
    s.o_fx2 = take(half);
    s.o_fpart = take(part);
    s.o_fbnp = take(bnp);
    s.o_bh = take(act);
    s.o_bpart = take(part);
    s.o_bbnp = take(bnp);
    s.o_dh = take(act);
    // weight-gradient splits of the front conv (rows strided over ~2 workgroups per CU)
    {
      const int ktot = s.R * s.R * s.Cin;
      const int bo = s.C <= 32 ? 32 : 64;
      const int wt = ((ktot + 63) / 64) * ((s.C + bo - 1) / bo);
      int sp = std::max(1, 512 / std::max(1, wt));
      long rps = (s.M + sp - 1) / sp;
      rps = std::max<long>(rps, 512);
      rps = (rps + 31) / 32 * 32;
      s.wsplits = static_cast<int>((s.M + rps - 1) / rps);
      s.wrows = static_cast<int>(rps);
      s.o_wpart = take(static_cast<size_t>(s.wsplits) * s.C * ktot * sizeof(float));
    }
    s.o_dtmp = s.first ? 0 : take(static_cast<size_t>(s.M) * s.Cin * esz);
    }  // front scratch
    if (s.has_blocks) {
      s.o_xr1 = take(half);
      s.o_xr2 = take(half);
      s.o_dx1 = take(half);
      s.o_dx2 = take(half);
    }
    if (!s.first) {
      const size_t in_half = static_cast<size_t>(s.Min) * (s.Cin / 2) * esz;
      for (int p = 0; p < 2; ++p)
        for (int h = 0; h < 2; ++h) s.o_msg[p][h] = take(in_half);
      if (!s.has_front)
        for (int p = 0; p < 2; ++p)
          for (int h = 0; h < 2; ++h) s.o_xmsg[p][h] = take(in_half);
    }
    if (s.last) {
      s.o_y1 = take(half);
      s.o_y2 = take(half);
      s.o_g1 = take(half);
      s.o_g2 = take(half);
      s.o_pooled = take(static_cast<size_t>(d.n) * s.C * sizeof(float));
      s.o_dlogits = take(static_cast<size_t>(d.n) * k * sizeof(float));
      s.o_lossn = take(static_cast<size_t>(d.n) * sizeof(float));
    }
    if (s.first) s.o_labels = take(static_cast<size_t>(J + 1) * d.n * sizeof(int32_t));
    cur = nullptr;
  }
  cur = &st[0].mem[MEM_SCRATCH];
  o_probe_run = take(static_cast<size_t>(2 * n_bnch) * sizeof(float));
  ws_need = o;
  // caller-owned fp32 parameters, accumulator, momentum and running statistics;
  // the front copies' alignment slack goes to stage 0
  int64_t counted = 0;
  for (NetStage& s : st) {
    s.mem[MEM_PARAMS] = 3 * s.n_span * static_cast<int64_t>(sizeof(float)) +
                        2 * ((s.has_front ? s.C : 0) + (s.has_blocks ? s.blocks->n_bnch : 0)) *
                            static_cast<int64_t>(sizeof(float));
    for (int c = MEM_WEIGHT_COPIES; c < MEM_COUNT; ++c) counted += s.mem[c];
  }
  st[0].mem[MEM_SCRATCH] += static_cast<int64_t>(ws_need) - counted;
}

Net::~Net() {
  for (NetStage& s : st) {
    s.blocks.reset();  // its graphs reference its own streams only
    if (s.ev_f) (void)hipEventDestroy(s.ev_f);
    if (s.ev_b) (void)hipEventDestroy(s.ev_b);
    if (s.sf) (void)hipStreamDestroy(s.sf);
    if (s.sb) (void)hipStreamDestroy(s.sb);
  }
  if (ev_tick) (void)hipEventDestroy(ev_tick);
}

void Net::bind(float* th, float* gr, float* mo, float* rm, float* rv, void* w) {
  theta = th; grad = gr; mom = mo; rmean = rm; rvar = rv;
  ws = static_cast<char*>(w);
  for (NetStage& s : st) {
    if (!s.has_blocks) continue;
    s.blocks->bind(th + s.off_blocks, gr + s.off_blocks, mo + s.off_blocks, rm + s.run_blocks,
                   rv + s.run_blocks, ws + s.o_blocks_ws);
    s.blocks->opt = opt;
  }
}

hipError_t Net::ensure_streams() {
  hipError_t e;
  if (!ev_tick && (e = hipEventCreateWithFlags(&ev_tick, hipEventDisableTiming)) != hipSuccess) return e;
  for (NetStage& s : st) {
    if (s.sf) continue;
    if ((e = hipStreamCreateWithFlags(&s.sf, hipStreamNonBlocking)) != hipSuccess) return e;
    if ((e = hipStreamCreateWithFlags(&s.sb, hipStreamNonBlocking)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&s.ev_f, hipEventDisableTiming)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&s.ev_b, hipEventDisableTiming)) != hipSuccess) return e;
    if (s.has_blocks && (e = s.blocks->ensure_streams()) != hipSuccess) return e;
  }
  return hipSuccess;
}

void Net::sync_weights(hipStream_t q) {
  refresh_weights(dt, theta, front_segs, front_max_numel, ws + o_front_wfwd, ws + o_front_wdg, q);
  for (NetStage& s : st)
    if (s.has_blocks) s.blocks->sync_weights(q);
}

void* Net::ring_slot(const NetStage& s, int64_t m, int half) const {
  const int64_t idx = m < 0 ? s.ring_depth : m % s.ring_depth;
  char* slot = ws + s.o_ring + static_cast<size_t>(idx) * s.ring_slot_bytes;
  if (half == 0) return slot;
  return slot + static_cast<size_t>(s.Min) * (s.Cin / 2) * esz;
}

void* Net::ib_slot(const NetStage& s, int64_t m, int half) const {
  char* slot = ws + s.o_ib + static_cast<size_t>(m % s.buf_depth) * s.ib_slot_bytes;
  return slot + (half ? static_cast<size_t>(s.M) * (s.C / 2) * esz : 0);
}

char* Net::ps_slot(const NetStage& s, int64_t m) const {
  return ws + s.o_ps + static_cast<size_t>(m % s.buf_depth) * s.ps_slot_bytes;
}

void* Net::fwd_in(const NetStage& s, int64_t m, int half) const {
  if (s.has_front) return ring_slot(s, m, half);
  const size_t hb = static_cast<size_t>(s.M) * (s.C / 2) * esz;
  if (m < 0) return ws + s.o_bpin + (half ? hb : 0);
  return ws + s.o_fin[m & 1][half];
}

void* Net::fwd_dest(const NetStage& s, int64_t m, int half) const {
  if (s.last) return ws + (half ? s.o_y2 : s.o_y1);
  return fwd_in(st[s.j + 1], m, half);
}

// y for stage j's backward: the next stage's buffered input (a front), the
// reconstruction the next (reversible) stage sent back, or in the backprop
// pass (m < 0) the exact input the forward left.
const void* Net::bwd_y(const NetStage& s, int64_t m, int parity, int half) const {
  const NetStage& nx = st[s.j + 1];
  if (nx.has_front || m < 0) return fwd_in(nx, m, half);
  return ws + nx.o_xmsg[parity][half];
}

const void* Net::bwd_g(const NetStage& s, int parity, int half) const {
  return ws + st[s.j + 1].o_msg[parity][half];
}

FrontView Net::front_view(const NetStage& s) const {
  const WeightSeg& g = front_segs.seg[s.fseg];
  return FrontView{ws + o_front_wfwd + g.fwd_off * esz, ws + o_front_wdg + g.dg_off * esz,
                   theta + s.off_front_g, theta + s.off_front_b};
}

FrontView Net::stash_front_view(const NetStage& s, int64_t m) const {
  char* b = ps_slot(s, m);
  const float* th = reinterpret_cast<const float*>(b);
  return FrontView{b + s.ps_fwf, b + s.ps_fwd, th + (s.off_front_g - s.off_front_w),
                   th + (s.off_front_b - s.off_front_w)};
}

// Parameter buffer: the version the forward of micro-batch m is about to read
// (fp32 parameters and the compute copies), ahead of it on its stream.
void Net::stash_params(NetStage& s, int64_t m, hipStream_t q) {
  char* b = ps_slot(s, m);
  PETRA_HIP(hip_status, hipMemcpyAsync(b, theta + s.off_front_w, static_cast<size_t>(s.n_span) * sizeof(float),
                       hipMemcpyDeviceToDevice, q));
  if (s.has_blocks) {
    const Stage& blk = *s.blocks;
    const size_t cw = static_cast<size_t>(blk.n_conv) * esz;
    PETRA_HIP(hip_status, hipMemcpyAsync(b + s.ps_bwf, blk.wfwd, cw, hipMemcpyDeviceToDevice, q));
    PETRA_HIP(hip_status, hipMemcpyAsync(b + s.ps_bwd, blk.wdg, cw, hipMemcpyDeviceToDevice, q));
  }
  if (s.has_front) {
    const FrontView f = front_view(s);
    PETRA_HIP(hip_status, hipMemcpyAsync(b + s.ps_fwf, f.wf, static_cast<size_t>(s.C) * s.R * s.R * s.Cin * esz,
                         hipMemcpyDeviceToDevice, q));
    PETRA_HIP(hip_status, hipMemcpyAsync(b + s.ps_fwd, f.wd, static_cast<size_t>(s.n_front_w) * esz,
                         hipMemcpyDeviceToDevice, q));
  }
}

// Front conv + BN (+ ReLU on the images) into the two half-tensors the blocks read.
// keep: the conv output and its BN vectors go to the backward's buffers (and move
// the running statistics) so that front_backward can skip the recompute.
void Net::front_forward(NetStage& s, const void* in1, const void* in2, hipStream_t q, bool keep,
                        void* out1, void* out2) {
  ConvArgs a{};
  a.src = in1;
  a.src2 = in2;
  a.c_split = in2 ? s.Cin / 2 : s.Cin;
  a.wt = ws + o_front_wfwd + front_segs.seg[s.fseg].fwd_off * esz;
  a.out = ws + (keep ? s.o_bh : s.o_fh);
  a.partials = at<float>(keep ? s.o_bpart : s.o_fpart);
  a.n = desc.n; a.h = s.Hin; a.w = s.Win; a.c_in = s.Cin; a.p = s.H; a.q = s.W; a.c_out = s.C;
  a.r = s.R; a.s = s.R; a.stride = s.stride; a.pad = s.pad; a.k_tot = s.R * s.R * s.Cin;
  a.m = static_cast<int>(s.M);
  conv_gemm(dt, a, EP_STATS, q);
  float* v = at<float>(keep ? s.o_bbnp : s.o_fbnp);
  bn_stats_finalize(static_cast<const float*>(a.partials), conv_row_tiles(dt, a, EP_STATS), s.C, s.M,
                    theta + s.off_front_g, theta + s.off_front_b, desc.bn_eps, v, v + s.C,
                    v + 2 * s.C, v + 3 * s.C, keep ? rmean + s.run_front : nullptr,
                    keep ? rvar + s.run_front : nullptr, desc.bn_momentum, q);
  bn_apply_split(dt, a.out, v, v + s.C, s.first ? 1 : 0, out1 ? out1 : ws + s.o_fx1,
                 out2 ? out2 : ws + s.o_fx2, s.M, s.C, q);
}

void Net::stage_forward(NetStage& s, int64_t m, hipStream_t q, bool keep, bool buffers) {
  const void* in1 = fwd_in(s, m, 0);
  const void* in2 = s.first ? nullptr : fwd_in(s, m, 1);
  if (buffers && s.ps_slot_bytes) stash_params(s, m, q);
  const void* b1 = in1;   // the blocks' input
  const void* b2 = in2;
  if (s.has_front) {
    void* f1 = s.has_blocks ? ws + s.o_fx1 : fwd_dest(s, m, 0);
    void* f2 = s.has_blocks ? ws + s.o_fx2 : fwd_dest(s, m, 1);
    front_forward(s, in1, in2, q, keep, f1, f2);
    b1 = f1;
    b2 = f2;
  }
  if (!s.has_blocks) return;
  if (buffers && s.ib_slot_bytes) {
    const size_t hb = static_cast<size_t>(s.M) * (s.C / 2) * esz;
    PETRA_HIP(hip_status, hipMemcpyAsync(ib_slot(s, m, 0), b1, hb, hipMemcpyDeviceToDevice, q));
    PETRA_HIP(hip_status, hipMemcpyAsync(ib_slot(s, m, 1), b2, hb, hipMemcpyDeviceToDevice, q));
  }
  Stage& blk = *s.blocks;
  void* y1 = fwd_dest(s, m, 0);
  void* y2 = fwd_dest(s, m, 1);
  if (blk.use_graphs)
    (void)blk.graphs.run({1, reinterpret_cast<uintptr_t>(b1), reinterpret_cast<uintptr_t>(y1)}, q,
                         [&](hipStream_t c) { blk.forward(b1, b2, y1, y2, c); }, 0);
  else
    blk.forward(b1, b2, y1, y2, q);
}

// Recompute the front layer from its buffered input (unless recompute is false:
// then front_forward(keep) left its output and BN vectors in place) and take its
// VJP given the gradient (d1, d2) of its output; writes the gradient message for
// stage j - 1.
void Net::front_backward(NetStage& s, const void* in1, const void* in2, const void* d1,
                         const void* d2, int parity, hipStream_t q, bool recompute,
                         const FrontView* fvp) {
  const float inv_k = 1.0f / static_cast<float>(std::max(1, opt.accum_k));
  const FrontView fv = fvp ? *fvp : front_view(s);
  ConvArgs a{};
  a.src = in1;
  a.src2 = in2;
  a.c_split = in2 ? s.Cin / 2 : s.Cin;
  a.wt = fv.wf;
  a.out = ws + s.o_bh;
  a.partials = at<float>(s.o_bpart);
  a.n = desc.n; a.h = s.Hin; a.w = s.Win; a.c_in = s.Cin; a.p = s.H; a.q = s.W; a.c_out = s.C;
  a.r = s.R; a.s = s.R; a.stride = s.stride; a.pad = s.pad; a.k_tot = s.R * s.R * s.Cin;
  a.m = static_cast<int>(s.M);
  float* v = at<float>(s.o_bbnp);
  float* scale = v;
  float* shift = v + s.C;
  float* mean = v + 2 * s.C;
  float* rstd = v + 3 * s.C;
  float* ca = v + 4 * s.C;
  float* cb = v + 5 * s.C;
  float* cc = v + 6 * s.C;
  if (recompute) {
    conv_gemm(dt, a, EP_STATS, q);
    bn_stats_finalize(at<float>(s.o_bpart), conv_row_tiles(dt, a, EP_STATS), s.C, s.M, fv.gamma,
                      fv.beta, desc.bn_eps, scale, shift, mean, rstd, rmean + s.run_front,
                      rvar + s.run_front, desc.bn_momentum, q);
  }
  const int relu = s.first ? 1 : 0;
  split_bwd_partials(dt, d1, d2, ws + s.o_bh, scale, shift, mean, rstd, relu,
                     at<float>(s.o_bpart), s.M, s.C, q);
  bn_bwd_finalize(at<float>(s.o_bpart), split_tiles(s.M, s.C), s.C, s.M, fv.gamma, mean, rstd,
                  inv_k, grad + s.off_front_g, grad + s.off_front_b, ca, cb, cc, q);
  split_bwd_apply(dt, d1, d2, ws + s.o_bh, scale, shift, ca, cb, cc, mean, relu, ws + s.o_dh,
                  s.M, s.C, q);
  // weight gradient
  WgradArgs w{};
  w.dh = ws + s.o_dh;
  w.src = in1;
  w.src2 = in2;
  w.c_split = a.c_split;
  w.partials = at<float>(s.o_wpart);
  w.n = desc.n; w.h = s.Hin; w.w = s.Win; w.c_in = s.Cin; w.p = s.H; w.q = s.W; w.c_out = s.C;
  w.r = s.R; w.s = s.R; w.stride = s.stride; w.pad = s.pad; w.k_tot = a.k_tot;
  w.m = static_cast<int>(s.M);
  w.splits = s.wsplits;
  w.rows_per_split = s.wrows;
  conv_wgrad(dt, w, q);
  if (s.Cin != s.cin_real)
    wgrad_reduce_pad(w.partials, w.splits, s.C, s.R * s.R, s.Cin, s.cin_real, inv_k,
                     grad + s.off_front_w, q);
  else
    wgrad_reduce(w.partials, w.splits, static_cast<long>(s.C) * a.k_tot, inv_k,
                 grad + s.off_front_w, q);
  if (s.first) return;  // the images need no gradient
  // input gradient of the 1x1 stride-2 conv: dh @ W on the output grid, then
  // scattered to the even pixels of the input grid (zero elsewhere)
  ConvArgs g{};
  g.src = ws + s.o_dh;
  g.c_split = s.C;
  g.wt = fv.wd;
  g.out = ws + s.o_dtmp;
  g.n = desc.n; g.h = s.H; g.w = s.W; g.c_in = s.C; g.p = s.H; g.q = s.W; g.c_out = s.Cin;
  g.r = 1; g.s = 1; g.stride = 1; g.pad = 0; g.k_tot = s.C; g.m = static_cast<int>(s.M);
  conv_gemm(dt, g, EP_RESID, q);
  scatter_stride2_split(dt, ws + s.o_dtmp, ws + s.o_msg[parity][0], ws + s.o_msg[parity][1],
                        desc.n, s.Hin, s.Win, s.Cin, q);
}

void Net::stage_update(NetStage& s, hipStream_t q) {
  if (s.n_decay)
    sgd_update(theta + s.off_decay, grad + s.off_decay, mom + s.off_decay, s.n_decay, s.n_decay,
               opt.lr, opt.momentum, opt.weight_decay, opt.nesterov, q);
  if (s.has_blocks) s.blocks->update_kernels(q);
  if (s.n_plain)
    sgd_update(theta + s.off_plain, grad + s.off_plain, mom + s.off_plain, s.n_plain, 0, opt.lr,
               opt.momentum, opt.weight_decay, opt.nesterov, q);
  if (!s.has_front) return;
  WeightSegTable one{};
  one.nseg = 1;
  one.seg[0] = front_segs.seg[s.fseg];
  refresh_weights(dt, theta, one, static_cast<int64_t>(s.C) * s.R * s.R * s.Cin, ws + o_front_wfwd,
                  ws + o_front_wdg, q);
}

// Loss head of the last stage on its block output (y1, y2): loss, the gradient
// halves o_g1/o_g2 and the linear layer's accumulated gradients.
void Net::head(NetStage& s, const void* y1, const void* y2, const int32_t* labels, float* loss,
               hipStream_t q) {
  head_forward_backward(dt, y1, y2, desc.n, s.H * s.W, s.C, theta + s.off_fc_w,
                        theta + s.off_fc_b, desc.classes, labels, at<float>(s.o_pooled),
                        at<float>(s.o_dlogits), at<float>(s.o_lossn), ws + s.o_g1, ws + s.o_g2,
                        q);
  const float inv_k = 1.0f / static_cast<float>(std::max(1, opt.accum_k));
  head_param_grads(at<float>(s.o_pooled), at<float>(s.o_dlogits), at<float>(s.o_lossn), desc.n,
                   s.C, desc.classes, inv_k, grad + s.off_fc_w, grad + s.off_fc_b, loss, q);
}

// Swaps the accumulator, the running statistics and the accumulation count
// of the net and its stages for the duration of a probe's enqueue: gradients
// land unscaled in gout, running-statistic moves in the probe sink.
struct Net::Redirect {
  Net& n;
  float* g;
  float* rm;
  float* rv;
  int k;
  Redirect(Net& net, float* gout) : n(net), g(net.grad), rm(net.rmean), rv(net.rvar),
                                    k(net.opt.accum_k) {
    float* sink = net.at<float>(net.o_probe_run);
    n.grad = gout;
    n.rmean = sink;
    n.rvar = sink + n.n_bnch;
    n.opt.accum_k = 1;
    for (NetStage& s : n.st) {
      if (!s.has_blocks) continue;
      s.blocks->grad = gout + s.off_blocks;
      s.blocks->rmean = sink + s.run_blocks;
      s.blocks->rvar = sink + n.n_bnch + s.run_blocks;
      s.blocks->opt.accum_k = 1;
    }
  }
  ~Redirect() {
    n.grad = g;
    n.rmean = rm;
    n.rvar = rv;
    n.opt.accum_k = k;
    for (NetStage& s : n.st) {
      if (!s.has_blocks) continue;
      s.blocks->grad = g + s.off_blocks;
      s.blocks->rmean = rm + s.run_blocks;
      s.blocks->rvar = rv + s.run_blocks;
      s.blocks->opt.accum_k = k;
    }
  }
};

void Net::backward_stage(NetStage& s, int64_t mb, int mode, int parity, hipStream_t q,
                         const void* by1, const void* by2, const void* bg1, const void* bg2,
                         hipStream_t side, bool recompute) {
  FrontView fv = s.has_front ? front_view(s) : FrontView{};
  const void* d1 = bg1;   // gradient of the front layer's output
  const void* d2 = bg2;
  if (s.has_blocks) {
    Stage& blk = *s.blocks;
    // a stage without front sends its reconstructed input and its input
    // gradient straight to stage j - 1
    void* xr1 = ws + (s.has_front ? s.o_xr1 : s.o_xmsg[parity][0]);
    void* xr2 = ws + (s.has_front ? s.o_xr2 : s.o_xmsg[parity][1]);
    void* dx1 = ws + (s.has_front ? s.o_dx1 : s.o_msg[parity][0]);
    void* dx2 = ws + (s.has_front ? s.o_dx2 : s.o_msg[parity][1]);
    if (mode == 0) {
      // PETRA: reconstruct the blocks' input from their output with the current
      // parameters and take the VJP there
      if (blk.use_graphs)
        (void)blk.graphs.run({2, reinterpret_cast<uintptr_t>(by1), reinterpret_cast<uintptr_t>(bg1)}, q,
                             [&](hipStream_t c) { blk.backward(by1, by2, bg1, bg2, xr1, xr2, dx1, dx2, c); },
                             1);
      else
        blk.backward(by1, by2, bg1, bg2, xr1, xr2, dx1, dx2, q, side);
    } else {
      // Variants: the VJP at the stored input (bit 0) or at the input
      // reconstructed with the current parameters, with the stashed parameters
      // (bit 1) or the current ones.  The blocks' output at that point is
      // recomputed, and the reversible backward runs from it.
      const void* u1 = s.ib_slot_bytes ? ib_slot(s, mb, 0) : nullptr;
      const void* u2 = s.ib_slot_bytes ? ib_slot(s, mb, 1) : nullptr;
      if (!(mode & 1)) {
        blk.reconstruct(by1, by2, ws + s.o_rx1, ws + s.o_rx2, q);
        u1 = ws + s.o_rx1;
        u2 = ws + s.o_rx2;
      }
      if (mode & 2) {
        char* b = ps_slot(s, mb);
        blk.set_view(reinterpret_cast<const float*>(b) + (s.off_blocks - s.off_front_w),
                     b + s.ps_bwf, b + s.ps_bwd);
        if (s.has_front) fv = stash_front_view(s, mb);
      }
      blk.forward_with(u1, u2, ws + s.o_ry1, ws + s.o_ry2, blk.sb[0], q);
      blk.backward(ws + s.o_ry1, ws + s.o_ry2, bg1, bg2, xr1, xr2, dx1, dx2, q);
      blk.reset_view();
    }
    d1 = dx1;
    d2 = dx2;
  } else if (mode & 2) {
    fv = stash_front_view(s, mb);
  }
  if (!s.has_front) return;
  const void* in1 = ring_slot(s, mb, 0);
  const void* in2 = s.first ? nullptr : ring_slot(s, mb, 1);
  front_backward(s, in1, in2, d1, d2, parity, q, recompute, &fv);
}

// The reversible-backpropagation pass over one micro-batch on stream q, on the
// extra input slot of every stage, the extra label slot and the message
// parity the next tick does not read.
void Net::backprop_pass(const void* images, const int32_t* labels, float* loss, bool update,
                        hipStream_t q) {
  const int par = static_cast<int>(t & 1);
  NetStage& s0 = st[0];
  int32_t* lab = at<int32_t>(s0.o_labels) + static_cast<size_t>(J) * desc.n;
  pad_channels8(dt, images, desc.c_img, ring_slot(s0, -1, 0), s0.Min, q);
  copy_i32(labels, lab, desc.n, q);
  for (NetStage& s : st) stage_forward(s, -1, q, /*keep=*/true, /*buffers=*/false);
  NetStage& sl = st[J - 1];
  head(sl, ws + sl.o_y1, ws + sl.o_y2, lab, loss, q);
  for (int j = J - 1; j >= 0; --j) {
    NetStage& s = st[j];
    const void *by1, *by2, *bg1, *bg2;
    if (s.last) {
      by1 = ws + s.o_y1; by2 = ws + s.o_y2; bg1 = ws + s.o_g1; bg2 = ws + s.o_g2;
    } else {
      by1 = bwd_y(s, -1, par, 0); by2 = bwd_y(s, -1, par, 1);
      bg1 = bwd_g(s, par, 0); bg2 = bwd_g(s, par, 1);
    }
    backward_stage(s, -1, 0, par, q, by1, by2, bg1, bg2, nullptr, /*recompute=*/false);
    if (!update) continue;
    if (count_and_due(s)) {
      // stage j's gradient is complete; stages below read only its message
      stage_update(s, q);
      if (s.has_blocks) s.blocks->mark_updated();
    }
  }
}

void Net::backprop_step(const void* images, const int32_t* labels, float* loss, hipStream_t q) {
  backprop_pass(images, labels, loss, true, q);
}

void Net::probe_backprop(const void* images, const int32_t* labels, float* gout, hipStream_t q) {
  Redirect r(*this, gout);
  PETRA_HIP(hip_status, hipMemsetAsync(gout, 0, static_cast<size_t>(n_params) * sizeof(float), q));
  backprop_pass(images, labels, nullptr, false, q);
}

void Net::probe_tick(int mode, float* gout, hipStream_t q) {
  Redirect r(*this, gout);
  PETRA_HIP(hip_status, hipMemsetAsync(gout, 0, static_cast<size_t>(n_params) * sizeof(float), q));
  const int64_t J2 = 2 * static_cast<int64_t>(J) - 2;
  const int par = static_cast<int>(t & 1);
  for (NetStage& s : st) {
    const int64_t mb = t - (J2 - s.j);
    if (mb < 0 || mb >= fed) continue;
    const void *by1, *by2, *bg1, *bg2;
    if (s.last) {
      // the last stage runs the forward of its micro-batch in the same tick
      stage_forward(s, mb, q, false, false);
      head(s, ws + s.o_y1, ws + s.o_y2, at<int32_t>(st[0].o_labels) + (mb % J) * desc.n, nullptr,
           q);
      by1 = ws + s.o_y1; by2 = ws + s.o_y2; bg1 = ws + s.o_g1; bg2 = ws + s.o_g2;
    } else {
      const int pm = static_cast<int>((t - 1) & 1);
      by1 = bwd_y(s, mb, pm, 0); by2 = bwd_y(s, mb, pm, 1);
      bg1 = bwd_g(s, pm, 0); bg2 = bwd_g(s, pm, 1);
    }
    backward_stage(s, mb, s.last ? 0 : mode, par, q, by1, by2, bg1, bg2);
  }
}

// Accumulation bookkeeping of a stage: a stage without blocks counts along
// with the network's optimizer setting (its own counter).
bool Net::count_and_due(NetStage& s) {
  if (s.has_blocks) {
    s.blocks->count_backward();
    return s.blocks->update_due();
  }
  ++s.bwd_count;
  const int k = std::max(1, opt.accum_k);
  return s.bwd_count % k == 0;
}

bool Net::tick(const void* images, const int32_t* labels, float* loss, hipStream_t caller) {
  const int64_t J2 = 2 * static_cast<int64_t>(J) - 2;
  if (images != nullptr) ++fed;   // micro-batch number t enters at this tick
  PETRA_HIP(hip_status, hipEventRecord(ev_tick, caller));
  bool wrote_loss = false;
  for (NetStage& s : st) {
    PETRA_HIP(hip_status, hipStreamWaitEvent(s.sf, ev_tick, 0));
    PETRA_HIP(hip_status, hipStreamWaitEvent(s.sb, ev_tick, 0));
  }
  for (NetStage& s : st) {
    const int64_t mf = t - s.j;
    const int64_t mb = t - (J2 - s.j);
    const bool do_f = mf >= 0 && mf < fed;
    const bool do_b = mb >= 0 && mb < fed;
    if (do_f) {
      hipStream_t q = s.sf;
      if (s.first) {
        pad_channels8(dt, images, desc.c_img, ring_slot(s, mf, 0), s.Min, q);
        copy_i32(labels, at<int32_t>(st[0].o_labels) + (mf % J) * desc.n, desc.n, q);
      }
      stage_forward(s, mf, q, /*keep=*/false, /*buffers=*/true);
      if (s.last) {
        head(s, ws + s.o_y1, ws + s.o_y2, at<int32_t>(st[0].o_labels) + (mf % J) * desc.n, loss, q);
        wrote_loss = loss != nullptr;
      }
    }
    if (do_b) {
      // the last stage continues on the stream of its own forward (same micro-batch)
      hipStream_t q = s.last ? s.sf : s.sb;
      const void *by1, *by2, *bg1, *bg2;
      if (s.last) {
        by1 = ws + s.o_y1; by2 = ws + s.o_y2; bg1 = ws + s.o_g1; bg2 = ws + s.o_g2;
      } else {
        const int par = static_cast<int>((t - 1) & 1);
        by1 = bwd_y(s, mb, par, 0); by2 = bwd_y(s, mb, par, 1);
        bg1 = bwd_g(s, par, 0); bg2 = bwd_g(s, par, 1);
      }
      // the last stage has no delay: every variant is the PETRA backward there.
      // (Handing deferred weight gradients to the forward stream, as the
      // single-stage step does, measured slower here: 3.27 vs 3.09 ms per tick,
      // the stages' streams are busy with each other's work.)
      backward_stage(s, mb, s.last ? 0 : bwd_mode, static_cast<int>(t & 1), q, by1, by2, bg1, bg2);
      if (count_and_due(s)) {
        // the update follows this stage's forward and backward of the tick (Eq. 5)
        if (q != s.sb) {
          PETRA_HIP(hip_status, hipEventRecord(s.ev_f, q));
          PETRA_HIP(hip_status, hipStreamWaitEvent(s.sb, s.ev_f, 0));
        } else if (do_f) {
          PETRA_HIP(hip_status, hipEventRecord(s.ev_f, s.sf));
          PETRA_HIP(hip_status, hipStreamWaitEvent(s.sb, s.ev_f, 0));
        }
        stage_update(s, s.sb);
        if (s.has_blocks) s.blocks->mark_updated();
      }
    }
  }
  for (NetStage& s : st) {
    PETRA_HIP(hip_status, hipEventRecord(s.ev_f, s.sf));
    PETRA_HIP(hip_status, hipEventRecord(s.ev_b, s.sb));
    PETRA_HIP(hip_status, hipStreamWaitEvent(caller, s.ev_f, 0));
    PETRA_HIP(hip_status, hipStreamWaitEvent(caller, s.ev_b, 0));
  }
  ++t;
  return wrote_loss;
}

}  // namespace petra
