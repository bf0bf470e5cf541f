// libpnn host side: plan construction (shape inference, validation, parameter / workspace
// layouts, level schedules) and the C-ABI entry points that enqueue the grouped kernels.
//
// Schedules.  Every node of a segment gets a level: 1 + the largest level of its inputs (slot 0
// has level 0).  A forward call walks the levels upwards and issues, per level, ONE grouped launch
// per kernel kind holding the nodes of that level of every segment in the call (for
// parareal_fine_fwd: all N sub-networks, Alg. para2's parallel loop).  A backward call walks the
// levels downwards (Alg. para3).
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <initializer_list>
#include <new>
#include <string>
#include <vector>

#include "pnn.h"
#include "pnn_internal.h"

using namespace pnn;

namespace {

constexpr size_t NONE = (size_t)-1;

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
inline long cdiv(long a, long b) { return (a + b - 1) / b; }

struct NodeP {
  int op, src, dst, bn, pool, k, stride, pad, cout, res;
  int level = 0;
  int cin = 0, H = 0, W = 0, Ho = 0, Wo = 0;
  size_t w_off = NONE, gw_off = NONE, wt_off = NONE;
  bool dgrad = false;      // data gradient needed in the backward
  bool first_of_two = false;
  bool resident = false;   // part of the segment's run of resident units (unit_fwd_kernel)
};

struct SlotP {
  int H = 0, W = 0, C = 0;
  long elems = 0;
  int producer = -1;
  int level = 0;
  int bn = -1;
  int res_consumer = -1;
  int direct_consumer = -1;
  std::vector<int> bn_consumers;
  size_t saved_off = NONE;
  size_t g_off = NONE;
};

struct BnP {
  int slot = 0, C = 0;
  size_t p_off = 0, gp_off = 0;
  size_t stats_off = 0;
  size_t part_off = 0;
  int fwd_tiles = 0, bwd_tiles = 0;
  size_t dbn_off = NONE, coef_off = NONE, datmp_off = NONE;
  bool bnact_consumer = false;
  bool defer_apply = false;  // dbn not stored: the apply pass recomputes it (see build_segment)
  bool bnsum = false;        // its backward sums come from bnsum_kernel (no data-gradient tile)
  int fwd_tiles_in = 0;      // coarse input BN: forward sums from the previous block's last
                             // convolution (coarse_fwd_all), in its row tiles; 0 = not chained
  int fwd_rows = 0;          // rows of the normalised tensor per forward partial row
  int fwd_rows_in = 0;       // the same for the chained sums
  size_t cnt_word = 0;       // its arrival counters (bn_fwd_fuse): word offset in the segment's block
};

struct SegP {
  int part = 0, index = 0;
  bool short_tiles = false;   // convolutions in short tiles (the coarse blocks: one problem a launch)
  int in_h = 0, in_w = 0, in_c = 0;
  std::vector<NodeP> nodes;
  std::vector<SlotP> slots;
  std::vector<BnP> bns;
  std::vector<bool> needs;
  int out = 0;
  int max_level = 0;
  size_t param_bytes = 0, grad_bytes = 0;
  size_t saved_base = 0, saved_bytes = 0;
  size_t scr_base = 0, scr_bytes = 0;
  size_t cnt_off = 0;          // the BN arrival counters of the segment (scratch, relative), words
  long cnt_words = 0;
  // run of bottleneck units the resident kernel can take (find_unit_run): its first node, unit
  // count, the levels it covers, its input slot and the first unit's offsets / per-unit strides
  int ru_node = -1, ru_n = 0, ru_lo = 0, ru_hi = 0, ru_xslot = 0;
  UnitJob ru_job{};
  unsigned ru_dw = 0, ru_dg = 0, ru_dz = 0, ru_ds = 0;
};

struct WgradGeom {
  int wr, tiles_co, tiles_k, splits, mchunk;
  bool halo3 = false;      // 3x3 / stride 1 / pad 1 through the halo kernel (tiles_k = Cg / 16)
  bool gemm = false;       // wide 3x3 / stride 1 / pad 1 bf16 through the GEMM kernel
  int gtc = 0, gtk = 0;    // its tile: output channels, filter columns (128 or 64)
};

}  // namespace

struct pnn_plan {
  int dtype = 0, es = 4;
  int B = 0, N = 0, classes = 0;
  int img_h = 0, img_w = 0, img_c = 0;
  std::vector<SegP> pre, fine, coarse;
  size_t saved_bytes = 0, scratch_bytes = 0;
  size_t wpart_off = 0, wpart_bytes = 0;
  size_t head_off = 0, head_bytes = 0;
  size_t sq_off = 0, sq_bytes = 0;
  // resident units: on / off (pnn_set_resident), workgroups that fit the device at once (queried
  // once, -1: not yet), scratch region: barrier words, then per fine segment its partial sums
  int resident_on = 0;
  int unit_cap = -1;
  size_t unit_off = 0, unit_part_stride = 0;
  size_t flags_off = 0;             // non-finite flags (PNN_NFLAGS uint32, scratch)
  // independent chains of the fine sub-networks: up to `streams` streams, the call's stream and
  // internal ones created by pnn_set_streams (default priority, non-blocking); compute calls never
  // create streams or events
  int streams = 1;
  std::vector<hipStream_t> side;
  std::vector<hipEvent_t> fj;          // fork / join events (no timing), used round robin
  size_t fj_next = 0;
  size_t wpart_stride = 0;             // one split-K partial region per chain
  // GEMM-kernel K-split partial tiles: one region per chain like the weight-gradient partials
  // (stride 0: no problem of the plan is split)
  size_t kpart_off = 0, kpart_stride = 0;
  size_t act_off = 0, act_stride = 0;   // activated GEMM inputs (act_materialize), per chain
  // timing of one kernel family
  int timing_family = 0;
  std::vector<hipEvent_t> ev;
  size_t ev_used = 0;
  double t_flops = 0.0, t_bytes = 0.0;
  long long t_launches = 0;
};

namespace {

// ------------------------------------------------------------------------------------------------
// plan construction
// ------------------------------------------------------------------------------------------------

// Weight-gradient tiling.  3x3 / stride 1 / pad 1 convolutions whose stages of W3 rows are whole
// image rows go to the halo kernel: 16 output channels x one 16-channel input block x 9 taps per
// workgroup, split-K in multiples of the stage.  Everything else: (16 wr) x 64 dW tiles, split-K
// over m in multiples of 128 rows into about 1024 workgroups (four per CU: a wide layer's few tiles
// would otherwise each walk hundreds of thousands of rows).
WgradGeom wgrad_geom(int Co, int K, long M);

WgradGeom wgrad_geom_node(const NodeP& n, int B, int es) {
  const long M = (long)B * n.Ho * n.Wo;
  const int K = n.k * n.k * n.cin;
  const int kc = es == 2 ? 256 : 128;               // stage rows of the halo kernel (W3Cfg::KC)
  const int ve = 16 / es;
  const long pq = (long)n.Ho * n.Wo;
  const bool whole_rows = kc % n.Wo == 0 && (pq % kc == 0 || kc % pq == 0);
  if (n.k == 3 && n.stride == 1 && n.pad == 1 && n.H == n.Ho && n.W == n.Wo && n.Wo % 8 == 0 &&
      n.cin % 16 == 0 && n.cout % 16 == 0 && whole_rows) {
    const long nimg = kc > pq ? kc / pq : 1;
    const long rows = kc > pq ? n.Ho : kc / n.Wo;
    if (nimg * (rows + 2) * (n.Wo + 2) * (16 / ve) <= 1024) {      // W3Cfg::HC halo chunks / thread
      WgradGeom g;
      g.halo3 = true;
      g.wr = 1;
      g.tiles_co = n.cout / 16;
      g.tiles_k = n.cin / 16;
      const long base = (long)g.tiles_co * g.tiles_k;
      long splits = std::max(1L, std::min(cdiv(M, 4L * kc), cdiv(256, base)));
      g.mchunk = (int)(cdiv(cdiv(M, splits), kc) * kc);
      g.splits = (int)cdiv(M, g.mchunk);
      return g;
    }
  }
  // wide 3x3 bf16 problems the halo kernel does not take: GEMM tiles of 128 (else 64) output
  // channels x 128 (else 64) filter columns (one tap's channels), split over m in 64-pixel stages
  // into about 512 workgroups (two per CU), at least 16 stages each
  if (es == 2 && n.k == 3 && n.stride == 1 && n.pad == 1 && n.H == n.Ho && n.W == n.Wo && n.cin % 64 == 0 &&
      n.cout % 64 == 0 && M < (1L << 30)) {
    WgradGeom g;
    g.gemm = true;
    g.wr = 0;
    g.gtc = n.cout % 128 == 0 ? 128 : 64;
    g.gtk = n.cin % 128 == 0 ? 128 : 64;
    g.tiles_co = n.cout / g.gtc;
    g.tiles_k = K / g.gtk;
    const long base = (long)g.tiles_co * g.tiles_k;
    const long splits = std::max(1L, std::min(cdiv(M, 16L * 64), cdiv(512, base)));
    g.mchunk = (int)(cdiv(cdiv(M, splits), 64) * 64);
    g.splits = (int)cdiv(M, g.mchunk);
    return g;
  }
  return wgrad_geom(n.cout, K, M);
}

WgradGeom wgrad_geom(int Co, int K, long M) {
  WgradGeom g;
  g.wr = (Co % 64 == 0) ? 4 : (Co % 32 == 0) ? 2 : 1;
  g.tiles_co = Co / (16 * g.wr);
  g.tiles_k = (int)cdiv(K, 64);
  const long base = (long)g.tiles_co * g.tiles_k;
  long splits = std::max(1L, std::min(cdiv(M, 512), cdiv(1024, base)));
  long mchunk = cdiv(cdiv(M, splits), 128) * 128;
  g.mchunk = (int)mchunk;
  g.splits = (int)cdiv(M, mchunk);
  return g;
}


// Problems of the streaming pointwise kernel: narrow (16-column tiles) forward 1x1 / stride 1 /
// pad 0 convolutions without a residual or an addend, and data gradients of such convolutions that
// store dbn and reduce the sums of their input BN when that BN has no other consumer (K <= PW_MAXK).
// The deferred-apply BNs' sums-only passes go to the BN-sum kernel.
bool pw_fwd_node(const SegP& S, const NodeP& n, int es) {
  return n.op == PNN_OP_CONV && n.k == 1 && n.stride == 1 && n.pad == 0 && n.cin % (16 / es) == 0 &&
         n.cin <= PW_MAXK && n.res < 0 && n.dst != S.out && n.cout % 16 == 0 && conv_wn(n.cout) == 1;
}
bool pw_bwd_node(const SegP& S, const NodeP& n, int es) {
  return n.op == PNN_OP_CONV && n.dgrad && n.k == 1 && n.stride == 1 && n.pad == 0 && n.bn >= 0 &&
         !S.bns[n.bn].defer_apply && S.slots[n.src].bn_consumers.size() == 1 && n.cout % (16 / es) == 0 &&
         n.cout <= PW_MAXK && n.cin % 16 == 0 && conv_wn(n.cin) == 1;
}
// bnsum_kernel rows per workgroup in tiles of BNSUM_TR: BNSUM_ROWS, or in short-tile segments
// halved while the launch has fewer than SHORT_TILES_BELOW workgroups
int bnsum_wm(long M, int ncol, bool short_ok) {
  int wm = BNSUM_ROWS / BNSUM_TR;
  if (short_ok)
    while (wm > 1 && cdiv(M, (long)BNSUM_TR * wm) * cdiv(ncol, 64) < SHORT_TILES_BELOW) wm >>= 1;
  return wm;
}

// 64-row tiles per streaming pointwise workgroup: 8, or 2 for short-tile segments when 8 would give
// under SHORT_TILES_BELOW workgroups
int pw_wm(long M, int ncol, bool short_ok) {
  const long tiles = (M + 64 * 8 - 1) / (64 * 8) * (ncol / 16);
  return short_ok && tiles < SHORT_TILES_BELOW ? 2 : 8;
}

// The weight gradient of a narrow pointwise data-gradient problem is formed by the same pw_kernel
// launch (EPI_PW_WGRAD) when every output channel row is a whole 16-row MFMA tile and its split-K
// partial rows (one per workgroup) fit the region reserved for the weight-gradient kernel's splits.
// Likewise the BN-sum pass of a deferred-apply BN (bnsum_kernel) for its consumer's weight gradient.
// Returns the partial rows (the launch's row tiles), or 0 when the weight gradient is not fused.
long wgrad_fused_rows(const SegP& S, const NodeP& n, int B, int es) {
  if (n.op != PNN_OP_CONV || !n.dgrad || n.bn < 0 || n.cout % 16 != 0) return 0;
  const long M = (long)B * n.Ho * n.Wo;
  long tiles_m = 0;
  if (pw_bwd_node(S, n, es))
    tiles_m = cdiv(M, (long)PW_TR * pw_wm(M, n.cin, S.short_tiles));
  else if (S.bns[n.bn].bnsum && n.k == 1 && n.stride == 1 && n.pad == 0)
    tiles_m = cdiv(M, (long)BNSUM_TR * bnsum_wm(M, n.cin, S.short_tiles));
  else
    return 0;
  const WgradGeom g = wgrad_geom_node(n, B, es);
  return !g.halo3 && !g.gemm && tiles_m <= g.splits ? tiles_m : 0;
}

pnn_status build_segment(const pnn_segment_desc& d, int part, int index, int B, int es, SegP& S) {
  S.part = part;
  S.index = index;
  S.short_tiles = part == 2;
  S.in_h = d.in_h;
  S.in_w = d.in_w;
  S.in_c = d.in_c;
  if (d.in_h <= 0 || d.in_w <= 0 || d.in_c <= 0 || d.n_nodes < 0 || d.n_bn < 0) return PNN_ERR_SHAPE;
  if (d.n_nodes > 0 && d.nodes == nullptr) return PNN_ERR_NULL;
  if (d.n_bn > 0 && d.bn_slot == nullptr) return PNN_ERR_NULL;
  int n_slots = 1;
  for (int i = 0; i < d.n_nodes; ++i) n_slots = std::max(n_slots, std::max(d.nodes[i].dst, d.nodes[i].src) + 1);
  if (d.out_slot < 0 || d.out_slot >= n_slots) return PNN_ERR_SHAPE;
  S.slots.assign(n_slots, SlotP());
  S.slots[0].H = d.in_h;
  S.slots[0].W = d.in_w;
  S.slots[0].C = d.in_c;
  std::vector<bool> made(n_slots, false);
  made[0] = true;
  S.bns.resize(d.n_bn);
  for (int b = 0; b < d.n_bn; ++b) {
    if (d.bn_slot[b] < 0 || d.bn_slot[b] >= n_slots) return PNN_ERR_SHAPE;
    S.bns[b].slot = d.bn_slot[b];
    if (S.slots[d.bn_slot[b]].bn != -1) return PNN_ERR_SHAPE;   // one BN per slot
    S.slots[d.bn_slot[b]].bn = b;
  }
  for (int i = 0; i < d.n_nodes; ++i) {
    const pnn_node_desc& x = d.nodes[i];
    NodeP n;
    n.op = x.op; n.src = x.src; n.dst = x.dst; n.bn = x.bn; n.pool = x.pool; n.k = x.k;
    n.stride = x.stride; n.pad = x.pad; n.cout = x.cout; n.res = x.res;
    if (n.src < 0 || n.src >= n_slots || !made[n.src]) return PNN_ERR_SHAPE;
    if (n.dst <= 0 || n.dst >= n_slots || made[n.dst]) return PNN_ERR_SHAPE;
    if (n.res >= n_slots || (n.res >= 0 && !made[n.res])) return PNN_ERR_SHAPE;
    if (n.bn >= d.n_bn || (n.bn >= 0 && S.bns[n.bn].slot != n.src)) return PNN_ERR_SHAPE;
    const SlotP& s = S.slots[n.src];
    n.cin = s.C; n.H = s.H; n.W = s.W;
    int oc = s.C;
    if (n.op == PNN_OP_CONV) {
      if (n.k != 1 && n.k != 3) return PNN_ERR_UNSUPPORTED;
      if (n.stride < 1 || n.stride > 2 || n.pad < 0 || n.pad >= n.k || n.cout <= 0) return PNN_ERR_SHAPE;
      if (n.cout % 16 != 0) return PNN_ERR_UNSUPPORTED;
      n.Ho = (s.H + 2 * n.pad - n.k) / n.stride + 1;
      n.Wo = (s.W + 2 * n.pad - n.k) / n.stride + 1;
      oc = n.cout;
    } else if (n.op == PNN_OP_BNACT) {
      if (n.bn < 0 || (n.pool != 0 && n.pool != 2)) return PNN_ERR_SHAPE;
      if (n.pool == 2 && (s.H % 2 || s.W % 2)) return PNN_ERR_UNSUPPORTED;
      n.Ho = n.pool ? s.H / 2 : s.H;
      n.Wo = n.pool ? s.W / 2 : s.W;
    } else if (n.op == PNN_OP_MAXPOOL3) {
      if (part != 0 || n.bn >= 0) return PNN_ERR_UNSUPPORTED;
      n.Ho = (s.H + 2 - 3) / 2 + 1;
      n.Wo = (s.W + 2 - 3) / 2 + 1;
    } else {
      return PNN_ERR_SHAPE;
    }
    if (n.Ho <= 0 || n.Wo <= 0) return PNN_ERR_SHAPE;
    SlotP& o = S.slots[n.dst];
    o.H = n.Ho; o.W = n.Wo; o.C = oc;
    o.producer = i;
    if (n.res >= 0) {
      const SlotP& r = S.slots[n.res];
      if (r.H != o.H || r.W != o.W || r.C != o.C) return PNN_ERR_SHAPE;
    }
    n.level = 1 + std::max(s.level, n.res >= 0 ? S.slots[n.res].level : 0);
    o.level = n.level;
    made[n.dst] = true;
    S.max_level = std::max(S.max_level, n.level);
    S.nodes.push_back(n);
  }
  if (!made[d.out_slot]) return PNN_ERR_SHAPE;
  S.out = d.out_slot;
  for (auto& sl : S.slots) sl.elems = (long)B * sl.H * sl.W * sl.C;
  // consumers
  for (int i = 0; i < (int)S.nodes.size(); ++i) {
    NodeP& n = S.nodes[i];
    SlotP& s = S.slots[n.src];
    if (n.res >= 0) {
      if (S.slots[n.res].res_consumer != -1) return PNN_ERR_UNSUPPORTED;
      S.slots[n.res].res_consumer = i;
    }
    if (n.op == PNN_OP_MAXPOOL3) continue;
    if (n.bn >= 0) {
      s.bn_consumers.push_back(i);
      if (n.op == PNN_OP_BNACT) S.bns[n.bn].bnact_consumer = true;
    } else {
      if (s.direct_consumer != -1) return PNN_ERR_UNSUPPORTED;
      s.direct_consumer = i;
    }
  }
  for (auto& b : S.bns) {
    if (b.slot != 0 && S.nodes[S.slots[b.slot].producer].op != PNN_OP_CONV) return PNN_ERR_UNSUPPORTED;
    if (S.slots[b.slot].C % 16 != 0 || S.slots[b.slot].C > 512) return PNN_ERR_UNSUPPORTED;
  }
  for (auto& sl : S.slots) {
    if (!sl.bn_consumers.empty() && sl.direct_consumer != -1) return PNN_ERR_UNSUPPORTED;
    if (sl.bn_consumers.size() > 2) return PNN_ERR_UNSUPPORTED;
    if (sl.bn != -1 && S.bns[sl.bn].bnact_consumer && sl.bn_consumers.size() != 1) return PNN_ERR_UNSUPPORTED;
  }
  const SlotP& so = S.slots[S.out];
  if (so.res_consumer != -1 || !so.bn_consumers.empty() || so.direct_consumer != -1) return PNN_ERR_UNSUPPORTED;
  if (part != 0 && S.out != 0) {
    const SlotP& s0 = S.slots[0];
    if (s0.bn_consumers.empty() && s0.direct_consumer == -1) return PNN_ERR_UNSUPPORTED;
  }
  // backward roles.  needs[s]: some parameter lies upstream of slot s (or the segment's input
  // gradient is wanted, for g^j and F^j), so dL/ds must be formed.
  S.needs.assign(n_slots, false);
  S.needs[0] = part != 0;
  for (auto& n : S.nodes)
    S.needs[n.dst] = S.needs[n.src] || (n.res >= 0 && S.needs[n.res]) || n.op == PNN_OP_CONV || n.bn >= 0;
  for (int i = 0; i < (int)S.nodes.size(); ++i) {
    NodeP& n = S.nodes[i];
    if (n.op == PNN_OP_MAXPOOL3 && S.needs[n.src]) return PNN_ERR_UNSUPPORTED;
    if (n.op != PNN_OP_CONV) continue;
    n.dgrad = S.needs[n.src] || n.bn >= 0;
    if (n.dgrad && n.cin % 16 != 0) return PNN_ERR_UNSUPPORTED;
  }
  for (auto& sl : S.slots) {
    if (sl.bn_consumers.size() == 2) {
      // the consumer reached first in the backward (higher level, then later node) stores fp32
      int a = sl.bn_consumers[0], b = sl.bn_consumers[1];
      const bool a_first = S.nodes[a].level > S.nodes[b].level ||
                           (S.nodes[a].level == S.nodes[b].level && a > b);
      S.nodes[a_first ? a : b].first_of_two = true;
    }
  }
  // BN backward without a stored dbn.  When the BN's only consumer is a pointwise convolution whose
  // output gradient has fewer than twice the BN's channels, its data-gradient pass only reduces the
  // BN sums, and a second pass of the same convolution forms dbn again and applies the BN backward:
  // re-reading the narrow output gradient costs fewer bytes than writing and re-reading dbn.
  for (auto& b : S.bns) {
    const SlotP& sl = S.slots[b.slot];
    if (sl.bn_consumers.size() != 1 || !S.needs[b.slot]) continue;
    const NodeP& n = S.nodes[sl.bn_consumers[0]];
    if (n.op != PNN_OP_CONV || !n.dgrad || n.k != 1 || n.stride != 1 || n.pad != 0) continue;
    if (n.cout % (16 / es) != 0 || n.cout >= 2 * n.cin) continue;
    b.defer_apply = true;
    b.bnsum = n.cout <= BNSUM_MAXK && n.cin % 16 == 0;
  }
  // parameter / gradient layout
  size_t po = 0, go = 0;
  for (auto& n : S.nodes) {
    if (n.op != PNN_OP_CONV) continue;
    const size_t cnt = (size_t)n.cout * n.k * n.k * n.cin;
    n.w_off = po;
    po = align256(po + cnt * es);
    n.gw_off = go;
    go = align256(go + cnt * 4);
  }
  for (auto& b : S.bns) {
    b.C = S.slots[b.slot].C;
    b.p_off = po;
    po = align256(po + (size_t)b.C * 8);
    b.gp_off = go;
    go = align256(go + (size_t)b.C * 8);
  }
  S.param_bytes = po;
  S.grad_bytes = go;
  // saved workspace (relative): intermediate slots and BN statistics
  size_t so_ = 0;
  for (int s = 1; s < (int)S.slots.size(); ++s) {
    if (s == S.out) continue;
    S.slots[s].saved_off = so_;
    so_ = align256(so_ + (size_t)S.slots[s].elems * es);
  }
  for (auto& b : S.bns) {
    b.stats_off = so_;
    so_ = align256(so_ + (size_t)b.C * 16);
  }
  S.saved_bytes = so_;
  // segment scratch (relative): BN partials / dbn / coefficients, slot gradients, filter transposes
  size_t sc = 0;
  for (auto& b : S.bns) {
    const SlotP& sl = S.slots[b.slot];
    const long M = (long)B * sl.H * sl.W;
    b.C = sl.C;
    // partial rows = tiles of the producing convolution: the forward one writing the slot, the
    // data gradient of the consumer that reduces the BN sums (the second of two)
    int kf = 1, kb = 1;
    bool pwf = false, pwb = false;
    if (sl.producer >= 0 && S.nodes[sl.producer].op == PNN_OP_CONV) {
      kf = S.nodes[sl.producer].k;
      pwf = pw_fwd_node(S, S.nodes[sl.producer], es);
    }
    for (int ci : sl.bn_consumers)
      if (!S.nodes[ci].first_of_two) {
        kb = S.nodes[ci].k;
        pwb = pw_bwd_node(S, S.nodes[ci], es);
      }
    const bool sh = S.short_tiles;
    const int pw_rows = 64 * pw_wm(M, b.C, sh);
    b.fwd_rows = b.slot == 0 ? COLSTAT_ROWS : pwf ? pw_rows : 64 * conv_rows_wm(kf, M, b.C, sh);
    b.fwd_tiles = (int)cdiv(M, b.fwd_rows);
    b.bwd_tiles = (int)cdiv(M, b.bnsum ? BNSUM_TR * bnsum_wm(M, b.C, sh) : pwb ? pw_rows : 64 * conv_rows_wm(kb, M, b.C, sh));
    if (b.bnact_consumer) {
      const NodeP& c = S.nodes[sl.bn_consumers[0]];
      b.bwd_tiles = (int)cdiv((long)B * c.Ho * c.Wo, BNACT_PIX);
    }
    int tiles = std::max(b.fwd_tiles, b.bwd_tiles);
    // a coarse block's input BN may take its forward sums from the previous block's last
    // convolution (coarse_fwd_all), in that convolution's row tiles of at least 64 rows
    if (part == 2 && b.slot == 0) tiles = std::max(tiles, (int)cdiv(M, 64));
    b.part_off = sc;
    sc = align256(sc + (size_t)tiles * 2 * b.C * 4);
    b.cnt_word = (size_t)S.cnt_words;
    S.cnt_words += bnf_words(b.C, tiles);
    b.coef_off = sc;
    sc = align256(sc + (size_t)b.C * 12);
    if (!sl.bn_consumers.empty() && !b.defer_apply) {
      b.dbn_off = sc;
      sc = align256(sc + (size_t)sl.elems * es);
    }
    if (sl.bn_consumers.size() == 2) {
      b.datmp_off = sc;
      sc = align256(sc + (size_t)sl.elems * 4);
    }
  }
  for (int s = 1; s < (int)S.slots.size(); ++s) {
    if (s == S.out) continue;
    SlotP& sl = S.slots[s];
    const bool alias = sl.bn_consumers.empty() && sl.direct_consumer == -1;
    if (alias || !S.needs[s]) continue;
    sl.g_off = sc;
    sc = align256(sc + (size_t)sl.elems * es);
  }
  for (auto& n : S.nodes) {
    if (n.op != PNN_OP_CONV || !n.dgrad) continue;
    n.wt_off = sc;
    sc = align256(sc + (size_t)n.cout * n.k * n.k * n.cin * es);
  }
  S.cnt_off = sc;
  sc = align256(sc + (size_t)S.cnt_words * 4);
  S.scr_bytes = sc;
  return PNN_OK;
}

// A pre-activation bottleneck unit at node i in the resident kernel's form: 1x1 squeeze C -> MID,
// 3x3 MID -> MID, 1x1 expand MID -> C with the unit input as residual, every convolution behind a
// BN of its input, stride 1, UNIT_H x UNIT_W maps; z1 and z2 feed only the next convolution, the
// unit input only the squeeze's BN and the residual; the output is the segment output or feeds a BN.
bool unit_at(const SegP& S, int i) {
  if (i < 0 || i + 2 >= (int)S.nodes.size()) return false;
  const NodeP &a = S.nodes[i], &b = S.nodes[i + 1], &c = S.nodes[i + 2];
  auto conv = [](const NodeP& n, int k, int cin, int cout) {
    return n.op == PNN_OP_CONV && n.k == k && n.stride == 1 && n.pad == (k - 1) / 2 && n.cin == cin &&
           n.cout == cout && n.bn >= 0;
  };
  if (!conv(a, 1, UNIT_C, UNIT_MID) || !conv(b, 3, UNIT_MID, UNIT_MID) || !conv(c, 1, UNIT_MID, UNIT_C)) return false;
  if (a.H != UNIT_H || a.W != UNIT_W || b.src != a.dst || c.src != b.dst || c.res != a.src || a.res >= 0 ||
      b.res >= 0)
    return false;
  const SlotP &x = S.slots[a.src], &z1 = S.slots[a.dst], &z2 = S.slots[b.dst], &o = S.slots[c.dst];
  if (x.bn_consumers.size() != 1 || x.res_consumer != i + 2 || x.direct_consumer != -1) return false;
  if (z1.bn_consumers.size() != 1 || z1.res_consumer != -1 || z1.direct_consumer != -1) return false;
  if (z2.bn_consumers.size() != 1 || z2.res_consumer != -1 || z2.direct_consumer != -1) return false;
  return c.dst == S.out || o.bn >= 0;
}

// The segment's first run of at least two consecutive resident-form units whose tensors sit at
// constant per-unit strides (so the kernel addresses unit u as the first unit plus u strides).
void find_unit_run(SegP& S) {
  const int nn = (int)S.nodes.size();
  for (int i0 = 0; i0 + 2 < nn; ++i0) {
    if (!unit_at(S, i0)) continue;
    auto offs = [&](int k, unsigned* o) {   // w1 w2 w3 g1 g2 g3 z1 z2 s1 s2 s3 xo
      const int i = i0 + 3 * k;
      const NodeP &a = S.nodes[i], &b = S.nodes[i + 1], &c = S.nodes[i + 2];
      const size_t v[12] = {a.w_off, b.w_off, c.w_off, S.bns[a.bn].p_off, S.bns[b.bn].p_off, S.bns[c.bn].p_off,
                            S.slots[a.dst].saved_off, S.slots[b.dst].saved_off, S.bns[a.bn].stats_off,
                            S.bns[b.bn].stats_off, S.bns[c.bn].stats_off, S.slots[c.dst].saved_off};
      for (int t = 0; t < 12; ++t) o[t] = v[t] == NONE ? 0xffffffffu : (unsigned)v[t];
      for (int t = 0; t < 12; ++t)
        if (v[t] != NONE && v[t] > 0xfffffff0u) return false;
      return true;
    };
    unsigned o0[12], ok_[12];
    if (!offs(0, o0)) return;
    int n = 1;
    unsigned st[12] = {0};
    while (unit_at(S, i0 + 3 * n) && S.nodes[i0 + 3 * n].src == S.nodes[i0 + 3 * n - 1].dst) {
      if (!offs(n, ok_)) break;
      if (n == 1) {
        for (int t = 0; t < 12; ++t) st[t] = ok_[t] - o0[t];
        if (st[0] != st[1] || st[1] != st[2] || st[3] != st[4] || st[4] != st[5] || st[6] != st[7] ||
            st[8] != st[9] || st[9] != st[10])
          break;
      } else {
        bool same = true;
        for (int t = 0; t < 11; ++t) same = same && ok_[t] == o0[t] + n * st[t];
        if (!same) break;
      }
      // the previous unit's output slot is this unit's input: saved at the slot stride
      if (S.slots[S.nodes[i0 + 3 * n - 1].dst].saved_off != (size_t)o0[6] + (size_t)(n - 1) * st[6] +
                                                              (size_t)(o0[11] - o0[6]))
        break;
      ++n;
    }
    if (n < 2) return;
    const NodeP& last = S.nodes[i0 + 3 * n - 1];
    UnitJob& J = S.ru_job;
    J.nu = n;
    J.w1 = o0[0]; J.w2 = o0[1]; J.w3 = o0[2];
    J.g1 = o0[3]; J.g2 = o0[4]; J.g3 = o0[5];
    J.z1 = o0[6]; J.z2 = o0[7]; J.xo = o0[11];
    J.s1 = o0[8]; J.s2 = o0[9]; J.s3 = o0[10];
    const SlotP& lo = S.slots[last.dst];
    J.gN = (last.dst != S.out && lo.bn >= 0) ? (unsigned)S.bns[lo.bn].p_off : 0xffffffffu;
    J.sN = (last.dst != S.out && lo.bn >= 0) ? (unsigned)S.bns[lo.bn].stats_off : 0xffffffffu;
    S.ru_dw = st[0]; S.ru_dg = st[3]; S.ru_dz = st[6]; S.ru_ds = st[8];
    S.ru_node = i0;
    S.ru_n = n;
    S.ru_lo = S.nodes[i0].level;
    S.ru_hi = last.level;
    S.ru_xslot = S.nodes[i0].src;
    for (int i = i0; i < i0 + 3 * n; ++i) S.nodes[i].resident = true;
    return;
  }
}

// wgrad partial bytes needed by every level of a set of segments at once (deferred weight gradients)
size_t wgrad_all_bytes(const std::vector<SegP>& segs, int B, int es) {
  size_t tot = 0;
  for (auto& s : segs)
    for (auto& n : s.nodes) {
      if (n.op != PNN_OP_CONV) continue;
      WgradGeom g = wgrad_geom_node(n, B, es);
      tot = align256(tot + (size_t)g.splits * n.cout * n.k * n.k * n.cin * 4);
    }
  return tot;
}

// wgrad partial bytes needed by one level of a set of segments run together
size_t wgrad_level_bytes(const std::vector<SegP>& segs, int B, int es) {
  int maxL = 0;
  for (auto& s : segs) maxL = std::max(maxL, s.max_level);
  size_t best = 0;
  for (int L = 1; L <= maxL; ++L) {
    size_t tot = 0;
    for (auto& s : segs)
      for (auto& n : s.nodes) {
        if (n.level != L || n.op != PNN_OP_CONV) continue;
        const int K = n.k * n.k * n.cin;
        WgradGeom g = wgrad_geom_node(n, B, es);
        tot = align256(tot + (size_t)g.splits * n.cout * K * 4);
      }
    best = std::max(best, tot);
  }
  return best;
}

bool same_shape(const SegP& a, int slot_a, int h, int w, int c) {
  const SlotP& s = a.slots[slot_a];
  return s.H == h && s.W == w && s.C == c;
}

// ------------------------------------------------------------------------------------------------
// call-time machinery
// ------------------------------------------------------------------------------------------------

struct Ptrs {
  const void* in = nullptr;
  void* out = nullptr;
  const void* params = nullptr;
  float* grads = nullptr;
  const void* ext = nullptr;
  const void* gout = nullptr;
  void* gin = nullptr;
  bool in_sums = false;               // forward: the input BN's sums are already in its partial rows
  const SegP* out_sums = nullptr;     // forward: the output's convolution also forms the sums of
                                      // this segment's input BN (the next coarse block)
  const void* out_params = nullptr;   // forward: that segment's parameters (its BN's gamma, beta)
  bool resident = false;              // forward: the segment's unit run goes to the resident kernel
};

struct Ctx {
  pnn_plan* plan;
  char* saved;
  char* scratch;
  hipStream_t stream;
  char* wpart = nullptr;   // split-K weight-gradient partials (nullptr: the plan's first region)
  char* kpart = nullptr;   // K-split GEMM partial tiles (nullptr: the plan's first region)
  char* act = nullptr;     // activated GEMM inputs (nullptr: the plan's first region)
};

inline char* cp(const void* p) { return (char*)const_cast<void*>(p); }

void* slot_ptr(const Ctx& c, const SegP& S, const Ptrs& p, int s) {
  if (s == 0) return const_cast<void*>(p.in);
  if (s == S.out) return p.out;
  return c.saved + S.saved_base + S.slots[s].saved_off;
}
float* stats_ptr(const Ctx& c, const SegP& S, int b) {
  return (float*)(c.saved + S.saved_base + S.bns[b].stats_off);
}
float* part_ptr(const Ctx& c, const SegP& S, int b) {
  return (float*)(c.scratch + S.scr_base + S.bns[b].part_off);
}
unsigned* cnt_ptr(const Ctx& c, const SegP& S, int b) {
  return (unsigned*)(c.scratch + S.scr_base + S.cnt_off) + S.bns[b].cnt_word;
}
// a forward producer of BN b's partial rows (EPI_STATS) also finalises its statistics
void set_bn_fuse(ConvProb& p, const Ctx& c, const SegP& S, int b, const void* params) {
  p.flags |= EPI_BN_FUSE;
  p.bn_cnt = cnt_ptr(c, S, b);
  p.bn_gamma = (const float*)(cp(params) + S.bns[b].p_off);
  p.bn_stats = stats_ptr(c, S, b);
}
void* grad_ptr(const Ctx& c, const SegP& S, const Ptrs& p, int s) {
  if (s == S.out) return const_cast<void*>(p.gout);
  if (s == 0) return p.gin;
  const SlotP& sl = S.slots[s];
  if (sl.g_off == NONE) return grad_ptr(c, S, p, S.nodes[sl.res_consumer].dst);  // residual-only slot
  return c.scratch + S.scr_base + sl.g_off;
}
void* skip_ptr(const Ctx& c, const SegP& S, const Ptrs& p, int s) {
  const SlotP& sl = S.slots[s];
  if (sl.res_consumer < 0) return nullptr;
  return grad_ptr(c, S, p, S.nodes[sl.res_consumer].dst);
}

struct Timer {
  pnn_plan* plan;
  int family;
  bool on;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  Timer(pnn_plan* p, int fam, hipStream_t s) : plan(p), family(fam) {
    on = p->timing_family == fam && p->ev_used + 2 <= p->ev.size();
    if (on) {
      e0 = p->ev[p->ev_used];
      e1 = p->ev[p->ev_used + 1];
      p->ev_used += 2;
      hipEventRecord(e0, s);
    }
  }
  void done(hipStream_t s, double flops, double bytes) {
    if (!on) return;
    hipEventRecord(e1, s);
    plan->t_flops += flops;
    plan->t_bytes += bytes;
    plan->t_launches += 1;
  }
};

// Chunk a problem list into grouped launches of at most PNN_MAXG problems.
template <typename Launch, typename Prob, typename TilesOf, typename Fire>
int grouped(std::vector<Prob>& probs, TilesOf tiles_of, Fire fire) {
  size_t i = 0;
  while (i < probs.size()) {
    Launch L;
    L.n = 0;
    int tiles = 0;
    size_t first = i;
    while (i < probs.size() && L.n < (int)(sizeof(L.p) / sizeof(L.p[0]))) {
      Prob pr = probs[i];
      pr.tile_begin = tiles;
      tiles += tiles_of(pr);
      if constexpr (HasTb<Launch>::value) L.tb[L.n] = pr.tile_begin;
      L.p[L.n++] = pr;
      ++i;
    }
    if constexpr (HasTb<Launch>::value) {
      static_assert(sizeof(L.tb) / sizeof(L.tb[0]) == sizeof(L.p) / sizeof(L.p[0]), "lookup table per problem");
      L.tb[0] = L.n;   // (the first problem begins at 0: the entry holds the count)
    }
    if (tiles > 0) {
      int e = fire(L, tiles, first);
      if (e) return PNN_ERR_HIP;
    }
  }
  return PNN_OK;
}

int fire_colred(std::vector<ColRedProb>& probs, hipStream_t s) {
  return grouped<ColRedLaunch>(
      probs, [](const ColRedProb& p) { return colred_tiles(p.ncols, p.mode, p.rl_log2); },
      [&](const ColRedLaunch& L, int tiles, size_t) { return launch_colred(L, tiles, s); });
}

ColRedProb bn_fwd_red(const float* part, int rows, int rowh, const float* gamma, float* stats, int C,
                      long count) {
  ColRedProb r;
  std::memset(&r, 0, sizeof(r));
  r.part = part;
  r.rows = rows;
  r.rowh = rowh;
  r.ncols = 2 * C;
  r.mode = RED_BN_FWD;
  r.gamma = gamma;
  r.beta = gamma + C;
  r.stats = stats;
  r.count = count;
  return r;
}

double conv_flops(const ConvProb& p) { return 2.0 * p.M * (double)p.ncol * p.K; }
double conv_bytes(const ConvProb& p, int es, int mode) {
  double b = (double)p.B * p.H * p.W * p.Cg * es + (double)p.ncol * p.K * es;
  const double mo = (double)p.M * p.ncol;
  if (mode == MODE_FWD) {
    b += mo * es * (1 + (p.res ? 1 : 0) + (p.ext ? 1 : 0));
  } else if (p.flags & EPI_STORE_F32) {
    b += mo * 4;
  } else if (p.flags & EPI_BN_APPLY) {
    b += mo * es * (2 + (p.res ? 1 : 0));
  } else if (p.flags & EPI_BN_MASK) {
    b += mo * es * ((p.flags & EPI_NO_STORE) ? 1 : 2) + ((p.flags & EPI_ACC_IN) ? mo * 4 : 0);
  } else {
    b += mo * es * (1 + (p.res ? 1 : 0));
  }
  return b;
}

int fire_conv_gk(const Ctx& c, std::vector<ConvProb>& probs, int mode, int gk, int wn, int wm) {
  pnn_plan* plan = c.plan;
  return grouped<ConvLaunch>(
      probs, [](const ConvProb& p) { return p.tiles_m * p.tiles_n * std::max(p.ksplit, 1); },
      [&](const ConvLaunch& L, int tiles, size_t) {
        double fl = 0, by = 0;
        for (int i = 0; i < L.n; ++i) {
          fl += conv_flops(L.p[i]);
          by += conv_bytes(L.p[i], plan->es, mode);
        }
        Timer t(plan, 1, c.stream);
        int e = gk >= 4 ? launch_gemm(L, tiles, mode, gk == 5 ? 64 : GEMM_BN, c.stream)
                        : launch_conv(L, tiles, plan->dtype, mode, gk, wn, wm, c.stream);
        t.done(c.stream, fl, by);
        return e;
      });
}

// A 3x3 / stride 1 / pad 1 problem whose row tiles are whole image rows, whose input rows plus
// halo fit CONV_HALO_BYTES of LDS and whose filter columns fit conv_halo_nkb(wn) K steps of registers.
bool halo_ok(const ConvProb& p, int es) {
  if (p.k != 3 || p.stride != 1 || p.pad != 1 || p.H != p.P || p.W != p.Q) return false;
  const int ve = 16 / es;
  if (p.K > 4 * ve * conv_halo_nkb(p.wn)) return false;
  const int bm = 64 * p.wm;
  const int pq = p.P * p.Q;
  if (bm % p.Q != 0 || (pq % bm != 0 && bm % pq != 0)) return false;
  const long nimg = bm > pq ? bm / pq : 1;
  const long rows = bm > pq ? p.P : bm / p.Q;
  const long ps = p.Cg + (long)conv_halo_pad(p.Cg / ve, p.Q) * ve;
  return nimg * (rows + 2) * (p.Q + 2) * ps * es <= CONV_HALO_BYTES;
}

// A 3x3 / stride 1 / pad 1 bf16 problem for the GEMM kernel: K steps of GEMM_BK channels within
// one tap, 128-row tiles (the tall tiles it would otherwise take), 128-column tiles where ncol
// allows them, else 64-column ones.  Returns the column tile width, 0 for another kernel.
int gemm_tn(const ConvProb& p, int es) {
  if (!(es == 2 && p.k == 3 && p.stride == 1 && p.pad == 1 && p.H == p.P && p.W == p.Q &&
        p.Cg % GEMM_BK == 0 && p.Cg <= CONV_PRO_MAXC && 64 * p.wm == GEMM_BM))
    return 0;
  return p.ncol % GEMM_BN == 0 ? GEMM_BN : p.ncol % 64 == 0 ? 64 : 0;
}

// K splits of the GEMM problems with fewer than GEMM_SPLIT_BELOW tiles (`small`: their tiles in
// one call): about GEMM_SPLIT_WG workgroups over all of them, GEMM_MIN_SPLIT_STEPS K steps each at
// least (1: no split)
int gemm_split(const ConvProb& q, long small) {
  if (small <= 0 || q.tiles_m * q.tiles_n >= GEMM_SPLIT_BELOW) return 1;
  const long s = std::min<long>({GEMM_MAX_SPLIT, GEMM_SPLIT_WG / small, (q.K / GEMM_BK) / GEMM_MIN_SPLIT_STEPS});
  return s >= 2 ? (int)s : 1;
}

// Gather kind of a convolution problem: 0 pointwise, 1 vector gather, 2 element-wise gather,
// 3 halo tile, 4 the GEMM kernel with 128-column tiles, 5 with 64-column tiles.
int gather_kind(const ConvProb& p, int es) {
  if (p.Cg % (16 / es) != 0) return 2;
  if (p.k == 1 && p.stride == 1 && p.pad == 0) return 0;
  const int tn = gemm_tn(p, es);
  if (tn != 0) return tn == GEMM_BN ? 4 : 5;
  if (halo_ok(p, es)) return 3;
  return 1;
}

// one grouped launch per (gather kind, column sub-tiles, tall / short tiles)
int fire_conv(const Ctx& c, std::vector<ConvProb>& probs, int mode) {
  std::vector<ConvProb> by[6][3][2];
  for (auto& p : probs) {
    const int w = p.wn == 1 ? 0 : p.wn == 2 ? 1 : 2;
    const int gk = gather_kind(p, c.plan->es);
    ConvProb q = p;
    if (gk >= 4) q.tiles_n = q.ncol / (gk == 4 ? GEMM_BN : 64);
    by[gk][w][p.wm == conv_wm(p.wn, false) ? 0 : 1].push_back(q);
  }
  // GEMM launches: the longest K first, so that the longest tiles start first; the problems with
  // few tiles split K (their partial tiles in the context's region, summed by a second pass)
  // 64-column GEMM launches with fewer tiles than compute units run at one tile's latency, where
  // the halo kernel's tile (its input read once into LDS) is the shorter: those go back to it
  for (int w = 0; w < 3; ++w)
    for (int t = 0; t < 2; ++t) {
      auto& v = by[5][w][t];
      long tiles = 0;
      bool halo = true;
      for (auto& q : v) {
        tiles += (long)q.tiles_m * q.tiles_n;
        halo = halo && halo_ok(q, c.plan->es);
      }
      if (tiles < GEMM_NARROW_MIN_TILES && halo) {
        by[3][w][t].insert(by[3][w][t].end(), v.begin(), v.end());
        v.clear();
      }
      std::stable_sort(v.begin(), v.end(), [](const ConvProb& a, const ConvProb& b) { return a.K > b.K; });
      for (auto& q : v) q.ksplit = 1;
    }
  long small = 0;
  for (auto& v : by[4])
    for (auto& t : v) {
      std::stable_sort(t.begin(), t.end(), [](const ConvProb& a, const ConvProb& b) { return a.K > b.K; });
      for (auto& q : t)
        if (q.tiles_m * q.tiles_n < GEMM_SPLIT_BELOW) small += q.tiles_m * q.tiles_n;
    }
  pnn_plan* plan = c.plan;
  char* region = c.kpart != nullptr ? c.kpart
                 : plan->kpart_stride != 0 ? c.scratch + plan->kpart_off : nullptr;
  std::vector<ConvProb> split;
  size_t koff = 0;
  for (auto& v : by[4])
    for (auto& t : v)
      for (auto& q : t) {
        q.ksplit = region != nullptr ? gemm_split(q, small) : 1;
        const size_t need = (size_t)q.ksplit * q.tiles_m * q.tiles_n * GEMM_BM * GEMM_BN * 4;
        if (q.ksplit < 2 || koff + need > plan->kpart_stride) {   // (the region holds them all)
          q.ksplit = 1;
          continue;
        }
        q.kpart = (float*)(region + koff);
        koff += need;
        split.push_back(q);
      }
  for (int gk = 0; gk < 6; ++gk)
    for (int w = 0; w < 3; ++w)
      for (int t = 0; t < 2; ++t) {
        if (by[gk][w][t].empty()) continue;
        int e = fire_conv_gk(c, by[gk][w][t], mode, gk, 1 << w, conv_wm(1 << w, t == 1));
        if (e) return e;
      }
  return grouped<ConvLaunch>(
      split, [](const ConvProb& p) { return p.tiles_m * p.tiles_n * (GEMM_BN / GEMM_RBN); },
      [&](const ConvLaunch& L, int tiles, size_t) {
        double by2 = 0;
        for (int i = 0; i < L.n; ++i)
          by2 += (double)L.p[i].ksplit * L.p[i].tiles_m * L.p[i].tiles_n * GEMM_BM * GEMM_BN * 4;
        Timer tm(plan, 1, c.stream);
        int e = launch_gemm_reduce(L, tiles, mode, c.stream);
        tm.done(c.stream, 0.0, by2);
        return e;
      });
}

// streaming pointwise problems: one grouped launch
int fire_pw(const Ctx& c, std::vector<ConvProb>& probs, int mode) {
  pnn_plan* plan = c.plan;
  return grouped<ConvLaunch>(
      probs, [](const ConvProb& p) { return p.tiles_m * p.tiles_n; },
      [&](const ConvLaunch& L, int tiles, size_t) {
        double fl = 0, by = 0;
        for (int i = 0; i < L.n; ++i) {
          fl += conv_flops(L.p[i]);
          by += conv_bytes(L.p[i], plan->es, mode);
        }
        Timer t(plan, 3, c.stream);
        int r = launch_pw(L, tiles, plan->dtype, mode, c.stream);
        t.done(c.stream, fl, by);
        return r;
      });
}

void set_pw_tiles(ConvProb& p, bool short_tiles) {
  p.wn = 1;
  p.wm = pw_wm(p.M, p.ncol, short_tiles);
  p.tiles_m = (int)cdiv(p.M, 64 * p.wm);
  p.tiles_n = p.ncol / 16;
}

ConvProb conv_common(const pnn_plan* plan, const NodeP& n) {
  ConvProb p;
  std::memset(&p, 0, sizeof(p));
  p.k = n.k;
  p.stride = n.stride;
  p.pad = n.pad;
  return p;
}

int log2_or(int v) {
  if (v <= 0 || (v & (v - 1))) return -1;
  int l = 0;
  while ((1 << l) < v) ++l;
  return l;
}

void set_tiles(ConvProb& p, bool short_tiles) {
  p.cg_log2 = log2_or(p.Cg);
  p.q_log2 = log2_or(p.Q);
  p.pq_log2 = log2_or(p.P * p.Q);
  p.wn = conv_wn(p.ncol);
  p.wm = conv_rows_wm(p.k, p.M, p.ncol, short_tiles);
  p.tiles_m = (int)cdiv(p.M, 64 * p.wm);
  p.tiles_n = p.ncol / (16 * p.wn);
}

// Whether some convolution of the plan, forward or data gradient, is a GEMM-kernel problem with
// fewer than GEMM_SPLIT_BELOW tiles (the problems fire_conv splits along K).
bool plan_splits_k(const pnn_plan* plan) {
  for (auto* v : {&plan->pre, &plan->fine, &plan->coarse})
    for (const SegP& S : *v)
      for (const NodeP& n : S.nodes) {
        if (n.op != PNN_OP_CONV) continue;
        for (int dir = 0; dir < 2; ++dir) {
          ConvProb p = conv_common(plan, n);
          p.B = plan->B;
          p.H = dir ? n.Ho : n.H; p.W = dir ? n.Wo : n.W; p.Cg = dir ? n.cout : n.cin;
          p.P = dir ? n.H : n.Ho; p.Q = dir ? n.W : n.Wo; p.ncol = dir ? n.cin : n.cout;
          p.M = plan->B * p.P * p.Q;
          p.K = n.k * n.k * p.Cg;
          set_tiles(p, S.short_tiles);
          if (gather_kind(p, plan->es) == 4 && cdiv(p.M, GEMM_BM) * (p.ncol / GEMM_BN) < GEMM_SPLIT_BELOW)
            return true;
        }
      }
  return false;
}

// A forward GEMM problem with a BN prologue whose input holds at least ACT_MIN_BYTES: its input is
// activated once, ReLU(BN(z)) by the BN-ReLU pass into a per-chain region, and the GEMM reads that
// without a prologue.  The prologue would activate every input element once per tap and column
// tile (9 x ncol / 128 times), which costs the forward GEMM a quarter of its MFMA rate on such
// layers; the pass costs two tensor passes at the HBM rate.  Results are bit-identical (the same
// fused multiply-add, ReLU and rounding).
constexpr long ACT_MIN_BYTES = 32L << 20;
bool act_materialize(const ConvProb& p, int es) {
  return p.pro != nullptr && gemm_tn(p, es) != 0 && (long)p.B * p.H * p.W * p.Cg * es >= ACT_MIN_BYTES;
}

// Likewise the input of a GEMM weight gradient with a BN prologue (the prologue there activates
// each input element once per tap and output-channel tile).
bool wgrad_act(const NodeP& n, int B, int es) {
  return n.bn >= 0 && wgrad_geom_node(n, B, es).gemm && (long)B * n.H * n.W * n.cin * es >= ACT_MIN_BYTES;
}

// the forward geometry of conv node n (its prologue pointer only marked)
ConvProb fwd_geom(const pnn_plan* plan, const SegP& S, const NodeP& n) {
  ConvProb p = conv_common(plan, n);
  p.B = plan->B; p.H = n.H; p.W = n.W; p.Cg = n.cin;
  p.P = n.Ho; p.Q = n.Wo; p.ncol = n.cout;
  p.M = plan->B * n.Ho * n.Wo;
  p.K = n.k * n.k * n.cin;
  p.pro = n.bn >= 0 ? (const float*)&S : nullptr;
  if (pw_fwd_node(S, n, plan->es)) set_pw_tiles(p, S.short_tiles);
  else set_tiles(p, S.short_tiles);
  return p;
}

// bytes of the activated GEMM inputs a forward level of these segments needs at once (the largest
// over the levels; a chain runs a subset of the segments)
size_t act_level_bytes(const pnn_plan* plan, const std::vector<SegP>& segs) {
  size_t best = 0;
  int maxL = 0;
  for (const SegP& S : segs)
    for (const NodeP& n : S.nodes) maxL = std::max(maxL, n.level);
  for (int L = 1; L <= maxL; ++L) {
    size_t b = 0, bw = 0;   // forward convolutions, weight gradients (wgrad_act) of the level
    for (const SegP& S : segs)
      for (const NodeP& n : S.nodes) {
        if (n.level != L || n.op != PNN_OP_CONV) continue;
        const ConvProb p = fwd_geom(plan, S, n);
        const size_t bytes = (size_t)p.B * p.H * p.W * p.Cg * plan->es;
        if (act_materialize(p, plan->es)) b = align256(b + bytes);
        if (wgrad_act(n, plan->B, plan->es)) bw = align256(bw + bytes);
      }
    best = std::max({best, b, bw});
  }
  return best;
}

// ------------------------------------------------------------------------------------------------
// forward of a set of segments
// ------------------------------------------------------------------------------------------------
int seg_max_level(const std::vector<const SegP*>& segs) {
  int maxL = 0;
  for (auto* s : segs) maxL = std::max(maxL, s->max_level);
  return maxL;
}

// Forward of a set of segments: run_fwd_begin (identity segments, statistics of BNs on the segment
// inputs), then run_fwd_level for L = 1 .. max level.
int run_fwd_begin(const Ctx& c, const std::vector<const SegP*>& segs, const std::vector<Ptrs>& ptrs) {
  pnn_plan* plan = c.plan;
  const int B = plan->B, es = plan->es;
  // identity segments
  for (size_t i = 0; i < segs.size(); ++i) {
    const SegP& S = *segs[i];
    if (S.nodes.empty() && ptrs[i].out != ptrs[i].in) {
      if (hipMemcpyAsync(ptrs[i].out, ptrs[i].in, (size_t)S.slots[0].elems * es,
                         hipMemcpyDeviceToDevice, c.stream) != hipSuccess)
        return PNN_ERR_HIP;
    }
  }
  // statistics of BN instances on segment inputs
  {
    std::vector<ColStatProb> cs;
    std::vector<ColRedProb> fw;
    for (size_t i = 0; i < segs.size(); ++i) {
      const SegP& S = *segs[i];
      const SlotP& s0 = S.slots[0];
      if (s0.bn < 0) continue;
      const BnP& b = S.bns[s0.bn];
      const bool chained = ptrs[i].in_sums && b.fwd_tiles_in > 0;
      const long M = (long)B * s0.H * s0.W;
      const long rows = chained ? b.fwd_tiles_in : cdiv(M, COLSTAT_ROWS);
      // few partial rows: the column statistics (or, chained, the previous block's last
      // convolution) finalise the statistics themselves (bn_fwd_fuse)
      const bool fuse = rows <= BNF_MAX_ROWS;
      if (!chained) {
        ColStatProb p;
        p.x = ptrs[i].in;
        p.part = part_ptr(c, S, s0.bn);
        p.gamma = (const float*)(cp(ptrs[i].params) + b.p_off);
        p.stats = stats_ptr(c, S, s0.bn);
        p.cnt = cnt_ptr(c, S, s0.bn);
        p.M = M;
        p.C = s0.C;
        p.fuse = fuse ? 1 : 0;
        cs.push_back(p);
      }
      if (!fuse)
        fw.push_back(bn_fwd_red(part_ptr(c, S, s0.bn), (int)rows, chained ? b.fwd_rows_in : b.fwd_rows,
                                (const float*)(cp(ptrs[i].params) + b.p_off), stats_ptr(c, S, s0.bn), b.C, M));
    }
    int e = grouped<ColStatLaunch>(
        cs, [](const ColStatProb& p) { return (int)cdiv(p.M, COLSTAT_ROWS); },
        [&](const ColStatLaunch& L, int tiles, size_t) { return launch_colstat(L, tiles, plan->dtype, c.stream); });
    if (e) return e;
    if (fire_colred(fw, c.stream)) return PNN_ERR_HIP;
  }
  return PNN_OK;
}

int run_fwd_level(const Ctx& c, const std::vector<const SegP*>& segs, const std::vector<Ptrs>& ptrs, int L) {
  pnn_plan* plan = c.plan;
  const int B = plan->B, es = plan->es;
  {
    std::vector<ConvProb> cv_vec, cv_gen, cv_pw;
    std::vector<BnActProb> ba, act;     // act: activated GEMM inputs, ahead of the convolutions
    std::vector<MaxPool3Prob> mp;
    std::vector<ColRedProb> fw;
    char* act_region = c.act != nullptr ? c.act : plan->act_stride != 0 ? c.scratch + plan->act_off : nullptr;
    size_t act_used = 0;
    // producers of BN partial rows that may finalise the statistics themselves (bn_fwd_fuse): the
    // problem (list, index), the BN and its parameters, and the column reduce it would need
    struct Cand {
      std::vector<ConvProb>* v;
      size_t i;
      const SegP* fs;
      int fb;
      const void* fparams;
      bool own;                       // the BN of the node's own output (else the next block's)
      ColRedProb red;
    };
    std::vector<Cand> cands;
    for (size_t i = 0; i < segs.size(); ++i) {
      const SegP& S = *segs[i];
      const Ptrs& P = ptrs[i];
      for (const NodeP& n : S.nodes) {
        if (n.level != L || (P.resident && n.resident)) continue;
        const SlotP& so = S.slots[n.dst];
        const void* ext = (n.dst == S.out) ? P.ext : nullptr;
        if (n.op == PNN_OP_CONV) {
          ConvProb p = conv_common(plan, n);
          p.in = slot_ptr(c, S, P, n.src);
          p.wmat = cp(P.params) + n.w_off;
          p.out = slot_ptr(c, S, P, n.dst);
          p.res = n.res >= 0 ? slot_ptr(c, S, P, n.res) : nullptr;
          p.ext = ext;
          p.pro = n.bn >= 0 ? stats_ptr(c, S, n.bn) + 2 * S.bns[n.bn].C : nullptr;
          const SegP* fs = nullptr;       // the BN whose partial rows this convolution writes
          int fb = -1;
          const void* fparams = nullptr;
          if (so.bn >= 0) {
            p.part = part_ptr(c, S, so.bn);
            p.flags = EPI_STATS;
            fs = &S; fb = so.bn; fparams = P.params;
          } else if (n.dst == S.out && P.out_sums != nullptr) {
            const SegP& nx = *P.out_sums;
            p.part = part_ptr(c, nx, nx.slots[0].bn);
            p.flags = EPI_STATS;
            fs = &nx; fb = nx.slots[0].bn; fparams = P.out_params;
          }
          p.B = B; p.H = n.H; p.W = n.W; p.Cg = n.cin;
          p.P = n.Ho; p.Q = n.Wo; p.ncol = n.cout;
          p.M = B * n.Ho * n.Wo;
          p.K = n.k * n.k * n.cin;
          const bool pwn = pw_fwd_node(S, n, es);
          if (pwn) set_pw_tiles(p, S.short_tiles);
          else set_tiles(p, S.short_tiles);
          const size_t abytes = (size_t)p.B * p.H * p.W * p.Cg * es;
          if (act_region != nullptr && act_materialize(p, es) && act_used + abytes <= plan->act_stride) {
            BnActProb a;
            std::memset(&a, 0, sizeof(a));
            a.z = p.in;
            a.out = act_region + act_used;
            a.stats = stats_ptr(c, S, n.bn);
            a.B = B; a.H = n.H; a.W = n.W; a.C = n.cin; a.pool = 0;
            a.n_out = (long)B * n.H * n.W;
            a.pix = bnact_fwd_pix(n.cin, es);
            act.push_back(a);
            act_used = align256(act_used + abytes);
            p.in = a.out;
            p.pro = nullptr;
          }
          std::vector<ConvProb>& dst = pwn ? cv_pw : (n.cin % (16 / es) == 0 ? cv_vec : cv_gen);
          dst.push_back(p);
          if (fs != nullptr) {
            Cand cd{&dst, dst.size() - 1, fs, fb, fparams, so.bn >= 0, {}};
            if (cd.own) {
              const BnP& b = S.bns[so.bn];
              cd.red = bn_fwd_red(part_ptr(c, S, so.bn), b.fwd_tiles, b.fwd_rows,
                                  (const float*)(cp(P.params) + b.p_off), stats_ptr(c, S, so.bn), b.C,
                                  (long)B * so.H * so.W);
            }
            cands.push_back(cd);
          }
        } else if (n.op == PNN_OP_BNACT) {
          BnActProb p;
          std::memset(&p, 0, sizeof(p));
          p.z = slot_ptr(c, S, P, n.src);
          p.out = slot_ptr(c, S, P, n.dst);
          p.res = n.res >= 0 ? slot_ptr(c, S, P, n.res) : nullptr;
          p.ext = ext;
          p.stats = stats_ptr(c, S, n.bn);
          p.B = B; p.H = n.H; p.W = n.W; p.C = n.cin; p.pool = n.pool;
          p.n_out = (long)B * n.Ho * n.Wo;
          p.pix = bnact_fwd_pix(n.cin, es);
          ba.push_back(p);
        } else {
          MaxPool3Prob p;
          p.x = slot_ptr(c, S, P, n.src);
          p.y = slot_ptr(c, S, P, n.dst);
          p.B = B; p.H = n.H; p.W = n.W; p.C = n.cin; p.Ho = n.Ho; p.Wo = n.Wo;
          const int ve = 16 / es;
          p.ve = (p.C % ve == 0 && (((uintptr_t)p.x | (uintptr_t)p.y) & 15) == 0) ? ve : 1;
          mp.push_back(p);
        }
        if (so.bn >= 0 && n.op != PNN_OP_CONV) {
          const BnP& b = S.bns[so.bn];
          const long cnt = (long)B * so.H * so.W;
          fw.push_back(bn_fwd_red(part_ptr(c, S, so.bn), b.fwd_tiles, b.fwd_rows,
                                  (const float*)(cp(P.params) + b.p_off), stats_ptr(c, S, so.bn), b.C, cnt));
        }
      }
    }
    // the level's producers finalise their BN statistics themselves when each has few partial rows
    // and the level's convolutions fit the device in one wave (there the finalisation replaces a
    // launch gap; in larger levels every workgroup's arrival would cost more than the launch); the
    // next block's input BN (chained) by its rows alone, as that block's call decides it
    long level_wg = 0;
    for (auto* v : {&cv_vec, &cv_gen, &cv_pw})
      for (const ConvProb& q : *v) level_wg += (long)q.tiles_m * q.tiles_n;
    for (Cand& cd : cands) {
      ConvProb& q = (*cd.v)[cd.i];
      const bool fuse = q.tiles_m <= BNF_MAX_ROWS && (!cd.own || level_wg <= BNF_MAX_WG);
      if (fuse) set_bn_fuse(q, c, *cd.fs, cd.fb, cd.fparams);
      else if (cd.own) fw.push_back(cd.red);
    }
    int e = grouped<BnActLaunch>(
        act, [](const BnActProb& p) { return (int)cdiv(p.n_out, p.pix); },
        [&](const BnActLaunch& Lx, int tiles, size_t) { return launch_bnact_fwd(Lx, tiles, plan->dtype, c.stream); });
    if (e) return e;
    if ((e = fire_conv(c, cv_vec, MODE_FWD))) return e;
    if ((e = fire_conv(c, cv_gen, MODE_FWD))) return e;
    if ((e = fire_pw(c, cv_pw, MODE_FWD))) return e;
    e = grouped<BnActLaunch>(
        ba, [](const BnActProb& p) { return (int)cdiv(p.n_out, p.pix); },
        [&](const BnActLaunch& Lx, int tiles, size_t) { return launch_bnact_fwd(Lx, tiles, plan->dtype, c.stream); });
    if (e) return e;
    e = grouped<MaxPool3Launch>(
        mp, [](const MaxPool3Prob& p) { return (int)cdiv((long)p.B * p.Ho * p.Wo * p.C, 256L * p.ve); },
        [&](const MaxPool3Launch& Lx, int tiles, size_t) { return launch_maxpool3(Lx, tiles, plan->dtype, c.stream); });
    if (e) return e;
    if (fire_colred(fw, c.stream)) return PNN_ERR_HIP;
  }
  return PNN_OK;
}

// The BN arrival counters of the segments a forward call uses set to zero, ahead of its launches
// (one grouped launch; the counters are left zero by the kernels that use them, so this only
// covers a scratch not yet used by this plan or one left by a failed call).
int clear_counters(const Ctx& c, const std::vector<const SegP*>& segs) {
  std::vector<ZeroProb> z;
  for (const SegP* S : segs)
    if (S->cnt_words > 0) {
      ZeroProb q;
      q.p = (unsigned*)(c.scratch + S->scr_base + S->cnt_off);
      q.words = (int)S->cnt_words;
      z.push_back(q);
    }
  return grouped<ZeroLaunch>(
      z, [](const ZeroProb& q) { return (int)cdiv(q.words, ZERO_WORDS); },
      [&](const ZeroLaunch& L, int tiles, size_t) { return launch_zero(L, tiles, c.stream); });
}

int run_fwd(const Ctx& c, const std::vector<const SegP*>& segs, const std::vector<Ptrs>& ptrs) {
  int e = run_fwd_begin(c, segs, ptrs);
  for (int L = 1, maxL = seg_max_level(segs); e == PNN_OK && L <= maxL; ++L) e = run_fwd_level(c, segs, ptrs, L);
  return e;
}

// ------------------------------------------------------------------------------------------------
// backward of a set of segments
// ------------------------------------------------------------------------------------------------
// data gradient of conv node n: gathers dL/d(n.dst) through the transposed filter; epilogue unset
ConvProb dgrad_base(const Ctx& c, const SegP& S, const Ptrs& P, const NodeP& n) {
  ConvProb p = conv_common(c.plan, n);
  p.in = grad_ptr(c, S, P, n.dst);
  p.wmat = c.scratch + S.scr_base + n.wt_off;
  p.B = c.plan->B; p.H = n.Ho; p.W = n.Wo; p.Cg = n.cout;
  p.P = n.H; p.Q = n.W; p.ncol = n.cin;
  p.M = c.plan->B * n.H * n.W;
  p.K = n.k * n.k * n.cout;
  return p;
}

void bn_bwd_finalize(const Ctx& c, const SegP& S, const Ptrs& P, int s, std::vector<ColRedProb>& fin,
                     std::vector<BnApplyProb>& app, std::vector<ConvProb>& rec) {
  const SlotP& sl = S.slots[s];
  if (sl.bn < 0 || sl.bn_consumers.empty()) return;
  const BnP& b = S.bns[sl.bn];
  ColRedProb f;
  std::memset(&f, 0, sizeof(f));
  f.part = part_ptr(c, S, sl.bn);
  f.rows = b.bwd_tiles;
  f.ncols = 2 * b.C;
  f.mode = RED_BN_BWD;
  f.gamma = (const float*)(cp(P.params) + b.p_off);
  f.stats = stats_ptr(c, S, sl.bn);
  f.dgamma = (float*)(cp(P.grads) + b.gp_off);
  f.dbeta = f.dgamma + b.C;
  f.coef = (float*)(c.scratch + S.scr_base + b.coef_off);
  f.count = (long)c.plan->B * sl.H * sl.W;
  fin.push_back(f);
  if (!S.needs[s]) return;
  if (b.defer_apply) {
    ConvProb p = dgrad_base(c, S, P, S.nodes[sl.bn_consumers[0]]);
    p.flags = EPI_BN_APPLY;
    p.zsrc = slot_ptr(c, S, P, s);
    p.bnst = f.stats;
    p.coef = f.coef;
    p.out = grad_ptr(c, S, P, s);
    p.res = skip_ptr(c, S, P, s);
    set_tiles(p, S.short_tiles);
    rec.push_back(p);
    return;
  }
  BnApplyProb a;
  a.dbn = c.scratch + S.scr_base + b.dbn_off;
  a.z = slot_ptr(c, S, P, s);
  a.skip = skip_ptr(c, S, P, s);
  a.out = grad_ptr(c, S, P, s);
  a.stats = f.stats;
  a.coef = f.coef;
  a.n = sl.elems;
  a.C = sl.C;
  app.push_back(a);
}

int fire_finalize(const Ctx& c, std::vector<ColRedProb>& fin, std::vector<BnApplyProb>& app,
                  std::vector<ConvProb>& rec) {
  if (fire_colred(fin, c.stream)) return PNN_ERR_HIP;
  int e = grouped<BnApplyLaunch>(
      app, [](const BnApplyProb& p) { return (int)cdiv(p.n, ELT_TILE); },
      [&](const BnApplyLaunch& L, int tiles, size_t) { return launch_bn_apply(L, tiles, c.plan->dtype, c.stream); });
  if (e) return e;
  return fire_conv(c, rec, MODE_BWD);
}

// Weight gradients of the convolutions at level L (every level when L < 0) of a set of segments,
// grouped by kernel variant; their split-K partial sums are appended to ``red`` (RED_SUM).  With
// ``fused``, the convolutions whose weight gradient their pointwise data-gradient or BN-sum launch
// forms (wgrad_fused_rows) only get their partial region and their reduction; ``fused`` lists them
// with that region.
using FusedWgrad = std::vector<std::pair<const NodeP*, float*>>;
int fire_wgrads(const Ctx& c, const std::vector<const SegP*>& segs, const std::vector<Ptrs>& ptrs, int L,
                std::vector<ColRedProb>& red, FusedWgrad* fused = nullptr) {
  pnn_plan* plan = c.plan;
  const int B = plan->B, es = plan->es;
  char* wpart = c.wpart != nullptr ? c.wpart : c.scratch + plan->wpart_off;
  std::vector<WgradProb> wg_vec, wg_gen, wg_h3, wg_pw, wg_gemm;
  std::vector<BnActProb> act;          // activated inputs of the GEMM weight gradients (wgrad_act)
  char* act_region = c.act != nullptr ? c.act : plan->act_stride != 0 ? c.scratch + plan->act_off : nullptr;
  size_t act_used = 0;
  size_t woff = 0;
  for (size_t i = 0; i < segs.size(); ++i) {
    const SegP& S = *segs[i];
    const Ptrs& P = ptrs[i];
    for (const NodeP& n : S.nodes) {
      if ((L >= 0 && n.level != L) || n.op != PNN_OP_CONV) continue;
      WgradProb p;
      std::memset(&p, 0, sizeof(p));
      p.g = grad_ptr(c, S, P, n.dst);
      p.in = slot_ptr(c, S, P, n.src);
      p.pro = n.bn >= 0 ? stats_ptr(c, S, n.bn) + 2 * S.bns[n.bn].C : nullptr;
      p.B = B; p.H = n.H; p.W = n.W; p.Cg = n.cin; p.P = n.Ho; p.Q = n.Wo; p.Co = n.cout;
      p.k = n.k; p.stride = n.stride; p.pad = n.pad;
      p.M = B * n.Ho * n.Wo;
      p.K = n.k * n.k * n.cin;
      WgradGeom g = wgrad_geom_node(n, B, es);
      p.wr = g.wr; p.tiles_co = g.tiles_co; p.tiles_k = g.tiles_k; p.splits = g.splits; p.mchunk = g.mchunk;
      p.gtc = g.gtc; p.gtk = g.gtk;
      const size_t abytes = (size_t)B * n.H * n.W * n.cin * es;
      if (act_region != nullptr && wgrad_act(n, B, es) && act_used + abytes <= plan->act_stride) {
        BnActProb a;
        std::memset(&a, 0, sizeof(a));
        a.z = p.in;
        a.out = act_region + act_used;
        a.stats = stats_ptr(c, S, n.bn);
        a.B = B; a.H = n.H; a.W = n.W; a.C = n.cin; a.pool = 0;
        a.n_out = (long)B * n.H * n.W;
        a.pix = bnact_fwd_pix(n.cin, es);
        act.push_back(a);
        act_used = align256(act_used + abytes);
        p.in = a.out;
        p.pro = nullptr;
      }
      p.cg_log2 = log2_or(p.Cg);
      p.q_log2 = log2_or(p.Q);
      p.pq_log2 = log2_or(p.P * p.Q);
      p.part = (float*)(wpart + woff);
      woff = align256(woff + (size_t)g.splits * p.Co * p.K * 4);
      int rows = g.splits;
      const long frows = fused != nullptr ? wgrad_fused_rows(S, n, B, es) : 0;
      if (frows > 0) {
        fused->push_back({&n, p.part});
        rows = (int)frows;
      } else {
        const bool vec = n.cin % (16 / es) == 0;
        const bool pw = vec && n.k == 1 && n.stride == 1 && n.pad == 0;
        (g.gemm ? wg_gemm : g.halo3 ? wg_h3 : pw ? wg_pw : vec ? wg_vec : wg_gen).push_back(p);
      }
      ColRedProb r;
      std::memset(&r, 0, sizeof(r));
      r.part = p.part;
      r.dst = (float*)(cp(P.grads) + n.gw_off);
      r.rows = rows;
      r.ncols = p.Co * p.K;
      r.mode = RED_SUM;
      r.rl_log2 = red_sum_rl_log2(r.rows);
      red.push_back(r);
    }
  }
  {
    const int e = grouped<BnActLaunch>(
        act, [](const BnActProb& q) { return (int)cdiv(q.n_out, q.pix); },
        [&](const BnActLaunch& Lx, int tiles, size_t) { return launch_bnact_fwd(Lx, tiles, plan->dtype, c.stream); });
    if (e) return e;
  }
  // the GEMM problems by tile shape (one launch per shape)
  std::vector<WgradProb> wg_gemm_by[4];
  for (const WgradProb& p : wg_gemm) wg_gemm_by[(p.gtc == 128 ? 0 : 2) + (p.gtk == 128 ? 0 : 1)].push_back(p);
  for (int v = 0; v < 8; ++v) {
    auto& list = v == 0 ? wg_vec : v == 1 ? wg_gen : v == 2 ? wg_h3 : v == 3 ? wg_pw : wg_gemm_by[v - 4];
    int e = grouped<WgradLaunch>(
        list, [](const WgradProb& p) { return p.tiles_co * p.tiles_k * p.splits; },
        [&](const WgradLaunch& Lx, int tiles, size_t) {
          double fl = 0, by = 0;
          for (int i = 0; i < Lx.n; ++i) {
            const WgradProb& p = Lx.p[i];
            fl += 2.0 * p.M * (double)p.Co * p.K;
            by += (double)p.M * p.Co * es + (double)p.B * p.H * p.W * p.Cg * es + (double)p.Co * p.K * 4;
          }
          Timer t(plan, 2, c.stream);
          int e2 = v == 2   ? launch_wgrad3(Lx, tiles, plan->dtype, c.stream)
                   : v >= 4 ? launch_wgrad_gemm(Lx, tiles, Lx.p[0].gtc, Lx.p[0].gtk, c.stream)
                            : launch_wgrad(Lx, tiles, plan->dtype, v == 0 ? WG_VEC : v == 1 ? WG_GEN : WG_PW,
                                           c.stream);
          t.done(c.stream, fl, by);
          return e2;
        });
    if (e) return e;
  }
  return PNN_OK;
}

// Backward of a set of segments run together, level by level.  wgrad = false leaves the weight
// gradients to a later fire_wgrads (the coarse chain defers them).
// Backward of a set of segments: run_bwd_begin (transposed filters), run_bwd_level for L = max
// level .. 1, run_bwd_end (gradient of the segment inputs).  The split-K weight-gradient sums of
// level L are reduced in the same launch as the BN backward finalisation of level L - 1
// (independent of it; `pending` carries them); level L - 1's weight gradient reuses the partial
// region only after that launch (stream order).
int run_bwd_begin(const Ctx& c, const std::vector<const SegP*>& segs, const std::vector<Ptrs>& ptrs) {
  pnn_plan* plan = c.plan;
  // filters of the data-gradient convolutions, [c_in][k][k][c_out]
  {
    std::vector<TransposeProb> tp;
    for (size_t i = 0; i < segs.size(); ++i) {
      const SegP& S = *segs[i];
      for (const NodeP& n : S.nodes) {
        if (n.op != PNN_OP_CONV || !n.dgrad) continue;
        TransposeProb p;
        p.w = cp(ptrs[i].params) + n.w_off;
        p.wt = c.scratch + S.scr_base + n.wt_off;
        p.O = n.cout;
        p.T = n.k * n.k;
        p.C = n.cin;
        tp.push_back(p);
      }
    }
    int e = grouped<TransposeLaunch>(
        tp, [](const TransposeProb& p) { return (int)(p.T * cdiv(p.O, 64) * cdiv(p.C, 64)); },
        [&](const TransposeLaunch& L, int tiles, size_t) { return launch_transpose(L, tiles, plan->dtype, c.stream); });
    if (e) return e;
  }
  return PNN_OK;
}

int run_bwd_level(const Ctx& c, const std::vector<const SegP*>& segs, const std::vector<Ptrs>& ptrs, int L,
                  bool wgrad, std::vector<ColRedProb>& pending) {
  pnn_plan* plan = c.plan;
  const int B = plan->B;
  {
    // A: gradients of the slots produced at this level (+ the previous level's split-K sums)
    {
      std::vector<ColRedProb> fin;
      std::vector<BnApplyProb> app;
      std::vector<ConvProb> rec;
      for (size_t i = 0; i < segs.size(); ++i) {
        const SegP& S = *segs[i];
        for (const NodeP& n : S.nodes)
          if (n.level == L && n.dst != S.out) bn_bwd_finalize(c, S, ptrs[i], n.dst, fin, app, rec);
      }
      fin.insert(fin.end(), pending.begin(), pending.end());
      pending.clear();
      int e = fire_finalize(c, fin, app, rec);
      if (e) return e;
    }
    // B + C: weight gradients (those of the narrow pointwise problems come with their data
    // gradients below)
    std::vector<ColRedProb> red;
    FusedWgrad fused;
    if (wgrad) {
      int e = fire_wgrads(c, segs, ptrs, L, red, &fused);
      if (e) return e;
    }
    pending = std::move(red);
    // D + E: data gradients (first of two BN consumers, then the rest) and bnact backward
    for (int phase = 0; phase < 2; ++phase) {
      std::vector<ConvProb> dg, bs, pw;
      std::vector<BnActProb> ba;
      for (size_t i = 0; i < segs.size(); ++i) {
        const SegP& S = *segs[i];
        const Ptrs& P = ptrs[i];
        for (const NodeP& n : S.nodes) {
          if (n.level != L) continue;
          if (n.op == PNN_OP_BNACT && phase == 1) {
            const BnP& b = S.bns[n.bn];
            BnActProb p;
            std::memset(&p, 0, sizeof(p));
            p.z = slot_ptr(c, S, P, n.src);
            p.out = c.scratch + S.scr_base + b.dbn_off;
            p.g = grad_ptr(c, S, P, n.dst);
            p.stats = stats_ptr(c, S, n.bn);
            p.part = part_ptr(c, S, n.bn);
            p.B = B; p.H = n.H; p.W = n.W; p.C = n.cin; p.pool = n.pool;
            p.n_out = (long)B * n.Ho * n.Wo;
            p.pix = BNACT_PIX;
            ba.push_back(p);
            continue;
          }
          if (n.op != PNN_OP_CONV || !n.dgrad) continue;
          if ((phase == 0) != n.first_of_two) continue;
          ConvProb p = dgrad_base(c, S, P, n);
          if (n.bn >= 0) {
            const BnP& b = S.bns[n.bn];
            if (n.first_of_two) {
              p.flags = EPI_STORE_F32;
              p.out32 = (float*)(c.scratch + S.scr_base + b.datmp_off);
            } else {
              p.flags = EPI_BN_MASK | (b.defer_apply ? EPI_NO_STORE : 0);
              if (b.bnsum) {           // sums only, by the streaming BN-sum kernel
                p.zsrc = slot_ptr(c, S, P, n.src);
                p.bnst = stats_ptr(c, S, n.bn);
                p.part = part_ptr(c, S, n.bn);
                p.wm = bnsum_wm(p.M, p.ncol, S.short_tiles);
                p.tiles_m = (int)cdiv(p.M, (long)BNSUM_TR * p.wm);
                for (const auto& f : fused)
                  if (f.first == &n) {
                    p.flags |= EPI_PW_WGRAD;
                    p.out32 = f.second;
                  }
                p.tiles_n = (int)cdiv(p.ncol, 64);
                bs.push_back(p);
                continue;
              }
              if (pw_bwd_node(S, n, plan->es)) {   // narrow: the streaming pointwise kernel
                p.out = c.scratch + S.scr_base + b.dbn_off;
                p.zsrc = slot_ptr(c, S, P, n.src);
                p.bnst = stats_ptr(c, S, n.bn);
                p.part = part_ptr(c, S, n.bn);
                for (const auto& f : fused)
                  if (f.first == &n) {
                    p.flags |= EPI_PW_WGRAD;
                    p.out32 = f.second;
                  }
                set_pw_tiles(p, S.short_tiles);
                pw.push_back(p);
                continue;
              }
              p.out = b.defer_apply ? nullptr : c.scratch + S.scr_base + b.dbn_off;
              p.zsrc = slot_ptr(c, S, P, n.src);
              p.bnst = stats_ptr(c, S, n.bn);
              p.part = part_ptr(c, S, n.bn);
              if (b.datmp_off != NONE) {
                p.flags |= EPI_ACC_IN;
                p.acc_in = (const float*)(c.scratch + S.scr_base + b.datmp_off);
              }
            }
          } else {
            p.out = grad_ptr(c, S, P, n.src);
            p.res = skip_ptr(c, S, P, n.src);
          }
          set_tiles(p, S.short_tiles);
          dg.push_back(p);
        }
      }
      int e = fire_conv(c, dg, MODE_BWD);
      if (e) return e;
      e = grouped<ConvLaunch>(
          bs, [](const ConvProb& p) { return p.tiles_m * p.tiles_n; },
          [&](const ConvLaunch& Lx, int tiles, size_t) {
            double by = 0;
            for (int j = 0; j < Lx.n; ++j)
              by += (double)Lx.p[j].M * (Lx.p[j].K + Lx.p[j].ncol) * plan->es;
            Timer t(plan, 3, c.stream);
            int r = launch_bnsum(Lx, tiles, plan->dtype, c.stream);
            t.done(c.stream, 0, by);
            return r;
          });
      if (e) return e;
      e = fire_pw(c, pw, MODE_BWD);
      if (e) return e;
      e = grouped<BnActLaunch>(
          ba, [](const BnActProb& p) { return (int)cdiv(p.n_out, p.pix); },
          [&](const BnActLaunch& Lx, int tiles, size_t) { return launch_bnact_bwd(Lx, tiles, plan->dtype, c.stream); });
      if (e) return e;
    }
  }
  return PNN_OK;
}

int run_bwd_end(const Ctx& c, const std::vector<const SegP*>& segs, const std::vector<Ptrs>& ptrs,
                std::vector<ColRedProb>& pending) {
  // gradient of the segment inputs (+ the last level's split-K sums)
  {
    std::vector<ColRedProb> fin = std::move(pending);
    std::vector<BnApplyProb> app;
    std::vector<ConvProb> rec;
    for (size_t i = 0; i < segs.size(); ++i) {
      const SegP& S = *segs[i];
      if (S.part == 0 || ptrs[i].gin == nullptr) continue;
      bn_bwd_finalize(c, S, ptrs[i], 0, fin, app, rec);
    }
    int e = fire_finalize(c, fin, app, rec);
    if (e) return e;
  }
  return PNN_OK;
}

// the levels and the input gradient, once run_bwd_begin's transposed filters are in place
int run_bwd_body(const Ctx& c, const std::vector<const SegP*>& segs, const std::vector<Ptrs>& ptrs,
                 bool wgrad) {
  std::vector<ColRedProb> pending;
  int e = PNN_OK;
  for (int L = seg_max_level(segs); e == PNN_OK && L >= 1; --L) e = run_bwd_level(c, segs, ptrs, L, wgrad, pending);
  return e == PNN_OK ? run_bwd_end(c, segs, ptrs, pending) : e;
}

int run_bwd(const Ctx& c, const std::vector<const SegP*>& segs, const std::vector<Ptrs>& ptrs,
            bool wgrad = true) {
  int e = run_bwd_begin(c, segs, ptrs);
  return e == PNN_OK ? run_bwd_body(c, segs, ptrs, wgrad) : e;
}

// ------------------------------------------------------------------------------------------------
// independent chains
// ------------------------------------------------------------------------------------------------
// The level schedule only orders nodes of one segment; segments are independent.  The fine
// segments are grouped by the spatial size of their input (the ResNet stage they start in), so
// that each group's levels launch one kernel variant; while streams are left, the group with the
// most work is halved.  Each group runs its levels on a stream of its own: level L of every group
// is enqueued before level L + 1, and the small launches of one group overlap the others'.  One
// fork (the side streams wait for the call's stream) and one join (the call's stream waits for
// them) per call.  Timed runs keep one stream.
struct Chains {
  std::vector<std::vector<const SegP*>> segs;
  std::vector<std::vector<Ptrs>> ptrs;
  std::vector<Ctx> ctx;
};

// Groups and their contexts: group g runs on the call's stream (g = 0) or side stream g - 1 and
// uses split-K partial region g + 1 (region 0 stays with the calls that do not chain).
int chains_group(const Ctx& c, const std::vector<const SegP*>& segs, const std::vector<Ptrs>& ptrs,
                 Chains& ch) {
  pnn_plan* p = c.plan;
  const int maxg = p->timing_family != 0 ? 1 : std::min(p->streams, (int)p->side.size() + 1);
  std::vector<long> keys;
  for (size_t i = 0; i < segs.size(); ++i) {
    const long key = (long)segs[i]->slots[0].H << 20 | segs[i]->slots[0].W;   // the stage
    size_t g = std::find(keys.begin(), keys.end(), key) - keys.begin();
    if (g == keys.size()) keys.push_back(key);
    g %= (size_t)maxg;
    if (g >= ch.segs.size()) {
      ch.segs.resize(g + 1);
      ch.ptrs.resize(g + 1);
    }
    ch.segs[g].push_back(segs[i]);
    ch.ptrs[g].push_back(ptrs[i]);
  }
  // streams left over: halve the group with the most saved activation bytes (its work)
  auto work = [&](size_t g) {
    size_t w = 0;
    for (auto* sp : ch.segs[g]) w += sp->saved_bytes;
    for (auto& pp : ch.ptrs[g])
      if (pp.resident) return (size_t)0;   // resident runs stay in one chain (one launch at a time)
    return w;
  };
  while ((int)ch.segs.size() < maxg) {
    size_t big = 0;
    for (size_t g = 1; g < ch.segs.size(); ++g)
      if (work(g) > work(big)) big = g;
    if (work(big) == 0) break;
    const size_t n = ch.segs[big].size();
    if (n < 2) break;
    ch.segs.emplace_back(ch.segs[big].begin() + n / 2, ch.segs[big].end());
    ch.ptrs.emplace_back(ch.ptrs[big].begin() + n / 2, ch.ptrs[big].end());
    ch.segs[big].resize(n / 2);
    ch.ptrs[big].resize(n / 2);
  }
  const int G = (int)ch.segs.size();
  for (int g = 0; g < G; ++g) {
    Ctx d = c;
    d.wpart = c.scratch + p->wpart_off + (size_t)(g + 1) * p->wpart_stride;
    if (p->kpart_stride != 0) d.kpart = c.scratch + p->kpart_off + (size_t)(g + 1) * p->kpart_stride;
    if (p->act_stride != 0) d.act = c.scratch + p->act_off + (size_t)(g + 1) * p->act_stride;
    ch.ctx.push_back(d);
  }
  if (G <= 1) return PNN_OK;
  for (int g = 1; g < G; ++g) ch.ctx[g].stream = p->side[g - 1];
  return PNN_OK;
}

// Side streams of groups [g0, g1) wait for everything enqueued on the call's stream so far.
int chains_wait(const Ctx& c, const Chains& ch, int g0, int g1) {
  if (g1 <= g0 || ch.ctx.size() <= 1) return PNN_OK;
  pnn_plan* p = c.plan;
  hipEvent_t e = p->fj[p->fj_next++ % p->fj.size()];
  if (hipEventRecord(e, c.stream) != hipSuccess) return PNN_ERR_HIP;
  for (int g = std::max(g0, 1); g < g1; ++g)
    if (hipStreamWaitEvent(ch.ctx[g].stream, e, 0) != hipSuccess) return PNN_ERR_HIP;
  return PNN_OK;
}

int chains_fork(const Ctx& c, const std::vector<const SegP*>& segs, const std::vector<Ptrs>& ptrs,
                Chains& ch) {
  int e = chains_group(c, segs, ptrs, ch);
  return e ? e : chains_wait(c, ch, 1, (int)ch.ctx.size());
}

int chains_join(const Ctx& c, const Chains& ch) {
  pnn_plan* p = c.plan;
  int st = PNN_OK;
  for (size_t g = 1; g < ch.ctx.size(); ++g) {
    hipEvent_t e = p->fj[p->fj_next++ % p->fj.size()];
    if (hipEventRecord(e, ch.ctx[g].stream) != hipSuccess || hipStreamWaitEvent(c.stream, e, 0) != hipSuccess)
      st = PNN_ERR_HIP;
  }
  return st;
}

// The resident kernel's launches for the unit runs of the segments flagged in ptrs: one workgroup
// per image, the segments packed in waves of at most plan->unit_cap workgroups (all of a launch's
// workgroups must be resident together; the launches follow each other on the one stream).
int fire_units(const Ctx& c, const std::vector<const SegP*>& segs, const std::vector<Ptrs>& ptrs) {
  pnn_plan* plan = c.plan;
  const int B = plan->B;
  unsigned* sync = (unsigned*)(c.scratch + plan->unit_off);
  UnitLaunch L;
  std::memset(&L, 0, sizeof(L));
  auto fire = [&]() -> int {
    if (L.n == 0) return PNN_OK;
    if (launch_unit_reset(sync, c.stream) || launch_unit_fwd(L, c.stream)) return (int)PNN_ERR_HIP;
    L.n = 0;
    L.nwg = 0;
    L.nu_max = 0;
    return (int)PNN_OK;
  };
  for (size_t i = 0; i < segs.size(); ++i) {
    const SegP& S = *segs[i];
    const Ptrs& P = ptrs[i];
    if (!P.resident) continue;
    if (L.n == UNIT_MAXJ || L.nwg + B > plan->unit_cap) {
      const int e = fire();
      if (e) return e;
    }
    L.B = B;
    L.dw = S.ru_dw; L.dg = S.ru_dg; L.dz = S.ru_dz; L.ds = S.ru_ds;
    L.sync = sync;
    UnitJob J = S.ru_job;
    J.x_in = slot_ptr(c, S, P, S.ru_xslot);
    J.params = cp(P.params);
    J.saved = c.saved + S.saved_base;
    J.y_out = P.out;
    J.part = (float*)(c.scratch + plan->unit_off + UNIT_SYNC_BYTES + (size_t)S.index * plan->unit_part_stride);
    J.wg_begin = L.nwg;
    L.j[L.n++] = J;
    L.nwg += B;
    L.nu_max = std::max(L.nu_max, J.nu);
  }
  return fire();
}

// Resident unit runs of one chain: the level from which they all can start (each run's own first
// level, the latest of them), after dropping the runs that would end before it.
int resident_level(const std::vector<const SegP*>& segs, std::vector<Ptrs>& ptrs) {
  int lf = 0;
  for (size_t i = 0; i < segs.size(); ++i)
    if (ptrs[i].resident) lf = std::max(lf, segs[i]->ru_lo);
  for (size_t i = 0; i < segs.size(); ++i)
    if (ptrs[i].resident && segs[i]->ru_hi < lf) ptrs[i].resident = false;
  return lf;
}

int run_fwd_chains(const Ctx& c, const std::vector<const SegP*>& segs, const std::vector<Ptrs>& ptrs) {
  Chains ch;
  int e = chains_fork(c, segs, ptrs, ch);
  const int G = (int)ch.segs.size();
  std::vector<int> lf(G, 0);
  for (int g = 0; g < G; ++g) lf[g] = resident_level(ch.segs[g], ch.ptrs[g]);
  for (int g = 0; e == PNN_OK && g < G; ++g) e = run_fwd_begin(ch.ctx[g], ch.segs[g], ch.ptrs[g]);
  for (int L = 1, maxL = seg_max_level(segs); e == PNN_OK && L <= maxL; ++L)
    for (int g = 0; e == PNN_OK && g < G; ++g) {
      if (L == lf[g]) e = fire_units(ch.ctx[g], ch.segs[g], ch.ptrs[g]);
      if (e == PNN_OK && L <= seg_max_level(ch.segs[g])) e = run_fwd_level(ch.ctx[g], ch.segs[g], ch.ptrs[g], L);
    }
  const int ej = chains_join(c, ch);
  return e != PNN_OK ? e : ej;
}

int run_bwd_chains(const Ctx& c, const std::vector<const SegP*>& segs, const std::vector<Ptrs>& ptrs) {
  Chains ch;
  int e = chains_fork(c, segs, ptrs, ch);
  const int G = (int)ch.segs.size();
  std::vector<std::vector<ColRedProb>> pending(G);
  for (int g = 0; e == PNN_OK && g < G; ++g) e = run_bwd_begin(ch.ctx[g], ch.segs[g], ch.ptrs[g]);
  for (int L = seg_max_level(segs); e == PNN_OK && L >= 1; --L)
    for (int g = 0; e == PNN_OK && g < G; ++g)
      if (L <= seg_max_level(ch.segs[g])) e = run_bwd_level(ch.ctx[g], ch.segs[g], ch.ptrs[g], L, true, pending[g]);
  for (int g = 0; e == PNN_OK && g < G; ++g) e = run_bwd_end(ch.ctx[g], ch.segs[g], ch.ptrs[g], pending[g]);
  const int ej = chains_join(c, ch);
  return e != PNN_OK ? e : ej;
}

// The resident kernel runs when enabled and one sub-network's batch fits the device at once (the
// occupancy, queried when it is turned on).
bool resident_ok(pnn_plan* plan) {
  if (!plan->resident_on || plan->dtype != PNN_BF16) return false;
  return plan->unit_cap >= plan->B;
}

bool ok_ctx(pnn_plan* plan, void* saved, void* scratch) {
  return plan != nullptr && (plan->saved_bytes == 0 || saved != nullptr) &&
         (plan->scratch_bytes == 0 || scratch != nullptr);
}

// Alignment rules of the interface: tensors and parameter / gradient buffers 16 bytes (the kernels
// move 16-byte chunks), workspaces 256 bytes.  NULL passes (the NULL checks come first).
inline bool al(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }
bool al16(std::initializer_list<const void*> ps) {
  for (const void* p : ps)
    if (!al(p, 16)) return false;
  return true;
}
bool al16n(const void* const* a, int j0, int j1) {
  for (int j = j0; j < j1; ++j)
    if (!al(a[j], 16)) return false;
  return true;
}
bool al_ws(const void* saved, const void* scratch) { return al(saved, 256) && al(scratch, 256); }

}  // namespace

// ================================================================================================
// C ABI
// ================================================================================================

extern "C" {

const char* pnn_status_string(pnn_status s) {
  switch (s) {
    case PNN_OK: return "ok";
    case PNN_ERR_NULL: return "a required pointer is NULL";
    case PNN_ERR_SHAPE: return "inconsistent shapes or node list";
    case PNN_ERR_DTYPE: return "unknown storage type";
    case PNN_ERR_WORKSPACE: return "unknown workspace kind";
    case PNN_ERR_UNSUPPORTED: return "network form not supported by this library";
    case PNN_ERR_HIP: return "a HIP call failed";
    case PNN_ERR_INDEX: return "index out of range";
    case PNN_ERR_ALIGN: return "a pointer is not aligned as the interface requires";
    case PNN_ERR_TOO_LARGE: return "the problem exceeds the fixed scratch of an allocation-free entry point";
    default: return "unknown status";
  }
}

pnn_status pnn_plan_create(const pnn_net_desc* d, pnn_plan** out) {
  if (d == nullptr || out == nullptr) return PNN_ERR_NULL;
  *out = nullptr;
  if (d->dtype != PNN_F32 && d->dtype != PNN_BF16) return PNN_ERR_DTYPE;
  if (d->n_sub < 1 || d->batch < 1 || d->n_classes < 1 || d->img_h < 1 || d->img_w < 1 || d->img_c < 1)
    return PNN_ERR_SHAPE;
  if (d->pre == nullptr || d->fine == nullptr || (d->n_sub > 1 && d->coarse == nullptr)) return PNN_ERR_NULL;
  pnn_plan* p = new (std::nothrow) pnn_plan();
  if (p == nullptr) return PNN_ERR_HIP;
  p->dtype = d->dtype;
  p->es = d->dtype == PNN_BF16 ? 2 : 4;
  p->B = d->batch;
  p->N = d->n_sub;
  p->classes = d->n_classes;
  p->img_h = d->img_h;
  p->img_w = d->img_w;
  p->img_c = d->img_c;
  const int N = d->n_sub;
  p->pre.resize(N);
  p->fine.resize(N);
  p->coarse.resize(N - 1);
  pnn_status st = PNN_OK;
  for (int j = 0; j < N && st == PNN_OK; ++j) st = build_segment(d->pre[j], 0, j, p->B, p->es, p->pre[j]);
  for (int j = 0; j < N && st == PNN_OK; ++j) st = build_segment(d->fine[j], 1, j, p->B, p->es, p->fine[j]);
  for (int j = 0; j < N - 1 && st == PNN_OK; ++j) st = build_segment(d->coarse[j], 2, j, p->B, p->es, p->coarse[j]);
  // shapes along the network: C^j -> g^j, g^j -> F^j -> X_{j+1}, r_j = y_j - x_{j+1}
  for (int j = 0; j < N && st == PNN_OK; ++j) {
    const SegP &pr = p->pre[j], &fi = p->fine[j];
    if (pr.in_h != d->img_h || pr.in_w != d->img_w || pr.in_c != d->img_c) st = PNN_ERR_SHAPE;
    const SlotP& po = pr.slots[pr.out];
    if (!same_shape(fi, 0, po.H, po.W, po.C)) st = PNN_ERR_SHAPE;
    if (j + 1 < N) {
      const SlotP& yo = fi.slots[fi.out];
      const SegP& cr = p->coarse[j];
      const SegP& f2 = p->fine[j + 1];
      const SlotP& y2 = f2.slots[f2.out];
      if (!same_shape(cr, 0, yo.H, yo.W, yo.C)) st = PNN_ERR_SHAPE;
      if (!same_shape(cr, cr.out, y2.H, y2.W, y2.C)) st = PNN_ERR_SHAPE;
      if (!same_shape(f2, 0, yo.H, yo.W, yo.C)) st = PNN_ERR_SHAPE;   // x_{j+1} in X_j
      if (cr.nodes.empty()) st = PNN_ERR_UNSUPPORTED;
    }
  }
  if (st != PNN_OK) {
    delete p;
    return st;
  }
  // coarse_fwd_all: the last convolution of block j - 1 also forms the forward sums of block j's
  // input BN (the same tensor), in that convolution's row tiles
  for (int j = 1; j + 1 < N; ++j) {
    SegP& nx = p->coarse[j];
    const SegP& pv = p->coarse[j - 1];
    const int bn = nx.slots[0].bn;
    if (bn < 0 || pv.slots[pv.out].bn >= 0) continue;
    const NodeP* prod = nullptr;
    for (const NodeP& n : pv.nodes)
      if (n.dst == pv.out) prod = &n;
    if (prod == nullptr || prod->op != PNN_OP_CONV || pw_fwd_node(pv, *prod, p->es)) continue;
    ConvProb t;
    std::memset(&t, 0, sizeof(t));
    t.k = prod->k; t.Cg = prod->cin; t.P = prod->Ho; t.Q = prod->Wo; t.ncol = prod->cout;
    t.M = p->B * prod->Ho * prod->Wo;
    set_tiles(t, pv.short_tiles);
    if (t.ncol == nx.bns[bn].C && t.tiles_m <= cdiv(t.M, 64)) {
      nx.bns[bn].fwd_tiles_in = t.tiles_m;
      nx.bns[bn].fwd_rows_in = 64 * t.wm;
    }
  }
  // workspace layout: saved = [pre | fine | coarse]; scratch = [shared | per segment]
  size_t sv = 0;
  for (auto* v : {&p->pre, &p->fine, &p->coarse})
    for (auto& s : *v) {
      s.saved_base = sv;
      sv = align256(sv + s.saved_bytes);
    }
  p->saved_bytes = sv;
  size_t wp = wgrad_level_bytes(p->fine, p->B, p->es);
  wp = std::max(wp, wgrad_level_bytes(p->pre, p->B, p->es));
  for (auto& s : p->coarse) wp = std::max(wp, wgrad_level_bytes(std::vector<SegP>{s}, p->B, p->es));
  wp = std::max(wp, wgrad_all_bytes(p->coarse, p->B, p->es));     // coarse_bwd_all
  wp = std::max(wp, wgrad_all_bytes(p->pre, p->B, p->es));        // pnn_pre_bwd, every level at once
  size_t sc = 0;
  p->wpart_off = sc;
  p->wpart_bytes = wp;
  p->wpart_stride = align256(wp);
  sc = align256(sc + p->wpart_stride * (PNN_MAX_CHAINS + 1));
  p->kpart_off = sc;
  p->kpart_stride = plan_splits_k(p) ? GEMM_KPART_BYTES : 0;
  sc = align256(sc + p->kpart_stride * (PNN_MAX_CHAINS + 1));
  size_t ab = act_level_bytes(p, p->fine);
  ab = std::max(ab, act_level_bytes(p, p->pre));
  for (auto& cs : p->coarse) ab = std::max(ab, act_level_bytes(p, std::vector<SegP>{cs}));
  p->act_off = sc;
  p->act_stride = ab;
  sc = align256(sc + p->act_stride * (PNN_MAX_CHAINS + 1));
  const SlotP& yo = p->fine[N - 1].slots[p->fine[N - 1].out];
  p->head_off = sc;
  p->head_bytes = (size_t)p->B * (yo.C + p->classes + 1) * 4;
  sc = align256(sc + p->head_bytes);
  long sqt = 0;
  for (int j = 0; j + 1 < N; ++j) sqt += cdiv(p->fine[j].slots[p->fine[j].out].elems, SUB_TILE);
  p->sq_off = sc;
  p->sq_bytes = (size_t)sqt * 4;
  sc = align256(sc + p->sq_bytes);
  p->flags_off = sc;
  sc = align256(sc + PNN_NFLAGS * 4);
  // resident units (bf16 storage): runs in the fine segments, their barrier words and partials
  if (p->dtype == PNN_BF16)
    for (auto& f : p->fine) find_unit_run(f);
  p->unit_off = sc;
  p->unit_part_stride = align256((size_t)p->B * (2 * UNIT_MID + UNIT_C) * 2 * 4);
  sc = align256(sc + UNIT_SYNC_BYTES + (size_t)N * p->unit_part_stride);
  for (auto* v : {&p->pre, &p->fine, &p->coarse})
    for (auto& s : *v) {
      s.scr_base = sc;
      sc = align256(sc + s.scr_bytes);
    }
  p->scratch_bytes = sc;
  *out = p;
  return PNN_OK;
}

void pnn_plan_destroy(pnn_plan* plan) {
  if (plan == nullptr) return;
  for (auto e : plan->ev) hipEventDestroy(e);
  for (auto e : plan->fj) hipEventDestroy(e);
  for (auto st : plan->side) hipStreamDestroy(st);
  delete plan;
}

pnn_status pnn_workspace_size(const pnn_plan* plan, int kind, size_t* bytes) {
  if (plan == nullptr || bytes == nullptr) return PNN_ERR_NULL;
  if (kind == PNN_WS_SAVED) *bytes = plan->saved_bytes;
  else if (kind == PNN_WS_SCRATCH) *bytes = plan->scratch_bytes;
  else return PNN_ERR_WORKSPACE;
  return PNN_OK;
}

pnn_status pnn_param_layout(const pnn_plan* plan, int part, int j, int grad, size_t* offsets, size_t* total) {
  if (plan == nullptr || total == nullptr) return PNN_ERR_NULL;
  const std::vector<SegP>* v = part == 0 ? &plan->pre : part == 1 ? &plan->fine : part == 2 ? &plan->coarse : nullptr;
  if (v == nullptr || j < 0 || j >= (int)v->size()) return PNN_ERR_INDEX;
  const SegP& S = (*v)[j];
  *total = grad ? S.grad_bytes : S.param_bytes;
  if (offsets) {
    const size_t nn = S.nodes.size();
    for (size_t i = 0; i < nn; ++i) offsets[i] = grad ? S.nodes[i].gw_off : S.nodes[i].w_off;
    for (size_t b = 0; b < S.bns.size(); ++b) {
      const size_t o = grad ? S.bns[b].gp_off : S.bns[b].p_off;
      offsets[nn + 2 * b] = o;
      offsets[nn + 2 * b + 1] = o + (size_t)S.bns[b].C * 4;
    }
  }
  return PNN_OK;
}

pnn_status pnn_tensor_shape(const pnn_plan* plan, int which, int j, int* h, int* w, int* c) {
  if (plan == nullptr || h == nullptr || w == nullptr || c == nullptr) return PNN_ERR_NULL;
  if (j < 0 || j >= plan->N || which < 0 || which > 1) return PNN_ERR_INDEX;
  const SegP& S = plan->fine[j];
  const SlotP& s = S.slots[which == 0 ? 0 : S.out];
  *h = s.H;
  *w = s.W;
  *c = s.C;
  return PNN_OK;
}

pnn_status pnn_pre_fwd(pnn_plan* plan, const void* image, void* const* x, const void* const* delta,
                       void* saved, void* scratch, void* stream) {
  if (!ok_ctx(plan, saved, scratch) || image == nullptr || x == nullptr) return PNN_ERR_NULL;
  if (!al_ws(saved, scratch)) return PNN_ERR_ALIGN;
  Ctx c{plan, (char*)saved, (char*)scratch, (hipStream_t)stream};
  std::vector<const SegP*> segs;
  std::vector<Ptrs> ptrs;
  for (int j = 0; j < plan->N; ++j) {
    const SegP& S = plan->pre[j];
    if (x[j] == nullptr) return PNN_ERR_NULL;
    if (S.param_bytes > 0 && (delta == nullptr || delta[j] == nullptr)) return PNN_ERR_NULL;
    if (!al16({image, x[j], delta ? delta[j] : nullptr})) return PNN_ERR_ALIGN;
    Ptrs p;
    p.in = image;
    p.out = x[j];
    p.params = delta ? delta[j] : nullptr;
    segs.push_back(&S);
    ptrs.push_back(p);
  }
  if (clear_counters(c, segs)) return PNN_ERR_HIP;
  return run_fwd(c, segs, ptrs);
}

pnn_status parareal_fine_fwd(pnn_plan* plan, const void* const* x, const void* const* phi, void* const* y,
                             void* saved, void* scratch, void* stream) {
  if (!ok_ctx(plan, saved, scratch) || x == nullptr || phi == nullptr || y == nullptr) return PNN_ERR_NULL;
  if (!al_ws(saved, scratch)) return PNN_ERR_ALIGN;
  Ctx c{plan, (char*)saved, (char*)scratch, (hipStream_t)stream};
  std::vector<const SegP*> segs;
  std::vector<Ptrs> ptrs;
  for (int j = 0; j < plan->N; ++j) {
    if (x[j] == nullptr || phi[j] == nullptr || y[j] == nullptr) return PNN_ERR_NULL;
    if (!al16({x[j], phi[j], y[j]})) return PNN_ERR_ALIGN;
    Ptrs p;
    p.in = x[j];
    p.out = y[j];
    p.params = phi[j];
    p.resident = resident_ok(plan) && plan->fine[j].ru_n >= 2;
    segs.push_back(&plan->fine[j]);
    ptrs.push_back(p);
  }
  if (clear_counters(c, segs)) return PNN_ERR_HIP;
  return run_fwd_chains(c, segs, ptrs);
}

pnn_status parareal_combine_fwd(pnn_plan* plan, const void* const* y, const void* const* x, void* const* r,
                                float* rnorm2, void* scratch, void* stream) {
  if (plan == nullptr) return PNN_ERR_NULL;
  if (plan->N == 1) return PNN_OK;
  if (y == nullptr || x == nullptr || r == nullptr) return PNN_ERR_NULL;
  if (rnorm2 != nullptr && scratch == nullptr) return PNN_ERR_NULL;
  if (!al(rnorm2, 4) || !al(scratch, 256)) return PNN_ERR_ALIGN;
  hipStream_t s = (hipStream_t)stream;
  std::vector<AxpyProb> pr;
  float* sq = rnorm2 ? (float*)((char*)scratch + plan->sq_off) : nullptr;
  unsigned* flag = scratch ? (unsigned*)((char*)scratch + plan->flags_off) : nullptr;
  long off = 0;
  for (int j = 0; j + 1 < plan->N; ++j) {
    if (y[j] == nullptr || x[j + 1] == nullptr || r[j] == nullptr) return PNN_ERR_NULL;
    if (!al16({y[j], x[j + 1], r[j]})) return PNN_ERR_ALIGN;
    AxpyProb p;
    p.a = y[j];
    p.b = x[j + 1];
    p.out = r[j];
    p.n = plan->fine[j].slots[plan->fine[j].out].elems;
    p.sq_part = sq ? sq + off : nullptr;
    off += cdiv(p.n, SUB_TILE);
    pr.push_back(p);
  }
  int e = grouped<AxpyLaunch>(
      pr, [](const AxpyProb& p) { return (int)cdiv(p.n, SUB_TILE); },
      [&](const AxpyLaunch& L, int tiles, size_t) {
        AxpyLaunch M = L;
        M.flag = flag;
        return launch_sub(M, tiles, plan->dtype, s);
      });
  if (e) return e;
  if (sq) {
    off = 0;
    for (int j = 0; j + 1 < plan->N; ++j) {
      const int t = (int)cdiv(pr[j].n, SUB_TILE);
      if (launch_sumsq(sq + off, t, rnorm2 + j, s)) return PNN_ERR_HIP;
      off += t;
    }
  }
  return PNN_OK;
}

pnn_status coarse_fwd(pnn_plan* plan, int j, const void* rt_j, const void* eta_j, const void* add,
                      void* rt_next, void* saved, void* scratch, void* stream) {
  if (!ok_ctx(plan, saved, scratch)) return PNN_ERR_NULL;
  if (j < 0 || j >= plan->N - 1) return PNN_ERR_INDEX;
  if (rt_j == nullptr || eta_j == nullptr || add == nullptr || rt_next == nullptr) return PNN_ERR_NULL;
  if (rt_j == rt_next) return PNN_ERR_SHAPE;
  if (!al16({rt_j, eta_j, add, rt_next}) || !al_ws(saved, scratch)) return PNN_ERR_ALIGN;
  Ctx c{plan, (char*)saved, (char*)scratch, (hipStream_t)stream};
  Ptrs p;
  p.in = rt_j;
  p.out = rt_next;
  p.params = eta_j;
  p.ext = add;
  if (clear_counters(c, {&plan->coarse[j]})) return PNN_ERR_HIP;
  return run_fwd(c, {&plan->coarse[j]}, {p});
}

pnn_status coarse_fwd_all(pnn_plan* plan, void* const* rt, const void* const* eta, const void* const* add,
                          void* saved, void* scratch, void* stream) {
  if (!ok_ctx(plan, saved, scratch)) return PNN_ERR_NULL;
  if (rt == nullptr || eta == nullptr || add == nullptr) return PNN_ERR_NULL;
  const int N = plan->N;
  if (N < 2) return PNN_OK;
  for (int j = 0; j < N; ++j)
    if (rt[j] == nullptr) return PNN_ERR_NULL;
  for (int j = 0; j + 1 < N; ++j) {
    if (eta[j] == nullptr || add[j] == nullptr) return PNN_ERR_NULL;
    if (rt[j] == rt[j + 1]) return PNN_ERR_SHAPE;
  }
  if (!al16n(rt, 0, N) || !al16n(eta, 0, N - 1) || !al16n(add, 0, N - 1) || !al_ws(saved, scratch))
    return PNN_ERR_ALIGN;
  Ctx c{plan, (char*)saved, (char*)scratch, (hipStream_t)stream};
  auto chained = [&](int j) {   // block j's input BN takes its sums from block j - 1
    const SegP& S = plan->coarse[j];
    return j > 0 && S.slots[0].bn >= 0 && S.bns[S.slots[0].bn].fwd_tiles_in > 0;
  };
  std::vector<const SegP*> all;
  for (int j = 0; j + 1 < N; ++j) all.push_back(&plan->coarse[j]);
  if (clear_counters(c, all)) return PNN_ERR_HIP;
  for (int j = 0; j + 1 < N; ++j) {
    Ptrs p;
    p.in = rt[j];
    p.out = rt[j + 1];
    p.params = eta[j];
    p.ext = add[j];
    p.in_sums = chained(j);
    p.out_sums = (j + 2 < N && chained(j + 1)) ? &plan->coarse[j + 1] : nullptr;
    p.out_params = p.out_sums != nullptr ? eta[j + 1] : nullptr;
    const int e = run_fwd(c, {&plan->coarse[j]}, {p});
    if (e) return e;
  }
  return PNN_OK;
}

}  // extern "C"

// head shape of a plan, for the allocation-free head entry point (noalloc.hip)
int pnn::head_geometry(const pnn_plan* p, int* B, int* HW, int* C, int* K, int* dtype) {
  if (p == nullptr) return PNN_ERR_NULL;
  const SegP& S = p->fine[p->N - 1];
  const SlotP& yo = S.slots[S.out];
  *B = p->B;
  *HW = yo.H * yo.W;
  *C = yo.C;
  *K = p->classes;
  *dtype = p->dtype;
  return PNN_OK;
}

extern "C" {

pnn_status pnn_head_fwd_bwd(pnn_plan* plan, const void* ytilde, const float* eps, const int32_t* labels,
                            float* logits, float* loss, void* D_N, float* deps, void* scratch, void* stream) {
  if (plan == nullptr || ytilde == nullptr || eps == nullptr || labels == nullptr || loss == nullptr ||
      D_N == nullptr || deps == nullptr || scratch == nullptr)
    return PNN_ERR_NULL;
  if (!al16({ytilde, eps, D_N, deps}) || !al(labels, 4) || !al(logits, 4) || !al(loss, 4) || !al(scratch, 256))
    return PNN_ERR_ALIGN;
  const SegP& S = plan->fine[plan->N - 1];
  const SlotP& yo = S.slots[S.out];
  if (plan->classes > 4096 || yo.C > 8192) return PNN_ERR_UNSUPPORTED;
  int e = launch_head(ytilde, eps, labels, logits, loss, D_N, deps,
                      (float*)((char*)scratch + plan->head_off), plan->B, yo.H * yo.W, yo.C,
                      plan->classes, plan->dtype, (unsigned*)((char*)scratch + plan->flags_off) + 1,
                      (hipStream_t)stream);
  return e ? PNN_ERR_HIP : PNN_OK;
}

pnn_status pnn_sgd_step(pnn_plan* plan, int part, void* const* params, const float* const* grads,
                        float* const* momentum, float* const* master, int master_init, float lr,
                        float mu, float weight_decay, int nesterov, void* stream) {
  if (plan == nullptr || params == nullptr || grads == nullptr || momentum == nullptr) return PNN_ERR_NULL;
  if (part < 0 || part > 3) return PNN_ERR_INDEX;
  const hipStream_t st = (hipStream_t)stream;
  // tensors of the part, segment by segment: (segment, parameter offset, gradient offset, count, f32)
  struct T { int seg; size_t po, go; long cnt; bool f32; };
  std::vector<T> ts;
  if (part == 3) {
    const SegP& S = plan->fine[plan->N - 1];
    const long C = S.slots[S.out].C;
    ts.push_back({0, 0, 0, (long)plan->classes * C + plan->classes, true});
  } else {
    const std::vector<SegP>& segs = part == 0 ? plan->pre : part == 1 ? plan->fine : plan->coarse;
    for (size_t j = 0; j < segs.size(); ++j) {
      const SegP& S = segs[j];
      for (const NodeP& n : S.nodes)
        if (n.op == PNN_OP_CONV) ts.push_back({(int)j, n.w_off, n.gw_off, (long)n.cout * n.k * n.k * n.cin, false});
      for (const BnP& b : S.bns) ts.push_back({(int)j, b.p_off, b.gp_off, 2L * b.C, true});
    }
  }
  for (const T& t : ts)
    if (params[t.seg] == nullptr || grads[t.seg] == nullptr || momentum[t.seg] == nullptr) return PNN_ERR_NULL;
  // the master copies of storage-type filters (bf16 plans, parts 0 - 2)
  const bool use_master = master != nullptr && plan->dtype == PNN_BF16 && part != 3;
  for (const T& t : ts) {
    if (use_master && !t.f32 && master[t.seg] == nullptr) return PNN_ERR_NULL;
    if (!al16({params[t.seg], grads[t.seg], momentum[t.seg], use_master ? master[t.seg] : nullptr}))
      return PNN_ERR_ALIGN;
  }
  // launches of at most SGD_MAXT tensors from at most SGD_MAXS consecutive segments
  size_t i = 0;
  while (i < ts.size()) {
    SgdLaunch L;
    std::memset(&L, 0, sizeof(L));
    L.lr = lr;
    L.mu = mu;
    L.wd = weight_decay;
    L.nesterov = nesterov != 0;
    L.init = master_init != 0;
    const int seg0 = ts[i].seg;
    int chunks = 0;
    while (i < ts.size() && L.nt < SGD_MAXT && ts[i].seg - seg0 < SGD_MAXS) {
      const T& t = ts[i++];
      if (t.cnt <= 0) continue;
      if (t.po > 0xffffffffu || t.go > 0xffffffffu || t.cnt > 0x7fffffffL) return PNN_ERR_UNSUPPORTED;
      const int ls = t.seg - seg0;
      L.p[ls] = params[t.seg];
      L.g[ls] = grads[t.seg];
      L.v[ls] = momentum[t.seg];
      L.m[ls] = use_master ? master[t.seg] : nullptr;
      SgdEnt& e = L.e[L.nt++];
      e.p_off = (uint32_t)t.po;
      e.g_off = (uint32_t)t.go;
      e.count = (uint32_t)t.cnt;
      e.chunk0 = (uint32_t)chunks;
      e.seg = (uint16_t)ls;
      e.f32 = t.f32 ? 1 : 0;
      chunks += (int)cdiv(t.cnt, SGD_CHUNK);
    }
    if (L.nt > 0 && launch_sgd(L, chunks, plan->dtype, st)) return PNN_ERR_HIP;
  }
  return PNN_OK;
}

pnn_status coarse_bwd(pnn_plan* plan, int j, const void* D_next, const void* rt_j, const void* eta_j,
                      const void* saved, void* D_j, float* deta_j, void* scratch, void* stream) {
  if (!ok_ctx(plan, const_cast<void*>(saved), scratch)) return PNN_ERR_NULL;
  if (j < 0 || j >= plan->N - 1) return PNN_ERR_INDEX;
  if (D_next == nullptr || rt_j == nullptr || eta_j == nullptr || D_j == nullptr || deta_j == nullptr)
    return PNN_ERR_NULL;
  if (D_j == D_next) return PNN_ERR_SHAPE;
  if (!al16({D_next, rt_j, eta_j, D_j, deta_j}) || !al_ws(saved, scratch)) return PNN_ERR_ALIGN;
  Ctx c{plan, (char*)const_cast<void*>(saved), (char*)scratch, (hipStream_t)stream};
  Ptrs p;
  p.in = rt_j;
  p.params = eta_j;
  p.grads = deta_j;
  p.gout = D_next;
  p.gin = D_j;
  return run_bwd(c, {&plan->coarse[j]}, {p});
}

pnn_status coarse_bwd_all(pnn_plan* plan, void* const* D, const void* const* rt, const void* const* eta,
                          const void* saved, float* const* deta, void* scratch, void* stream) {
  if (!ok_ctx(plan, const_cast<void*>(saved), scratch)) return PNN_ERR_NULL;
  if (D == nullptr || rt == nullptr || eta == nullptr || deta == nullptr) return PNN_ERR_NULL;
  const int N = plan->N;
  if (N < 2) return PNN_OK;
  for (int j = 0; j < N; ++j)
    if (D[j] == nullptr) return PNN_ERR_NULL;
  for (int j = 0; j < N - 1; ++j)
    if (rt[j] == nullptr || eta[j] == nullptr || deta[j] == nullptr) return PNN_ERR_NULL;
  if (!al16n(D, 0, N) || !al16n(rt, 0, N - 1) || !al16n(eta, 0, N - 1) ||
      !al16n((const void* const*)deta, 0, N - 1) || !al_ws(saved, scratch))
    return PNN_ERR_ALIGN;
  Ctx c{plan, (char*)const_cast<void*>(saved), (char*)scratch, (hipStream_t)stream};
  std::vector<const SegP*> segs;
  std::vector<Ptrs> ptrs;
  for (int j = N - 2; j >= 0; --j) {
    Ptrs p;
    p.in = rt[j];
    p.params = eta[j];
    p.grads = deta[j];
    p.gout = D[j + 1];
    p.gin = D[j];
    if (D[j] == D[j + 1]) return PNN_ERR_SHAPE;
    segs.push_back(&plan->coarse[j]);
    ptrs.push_back(p);
  }
  // every block's transposed filters in one grouped launch, then the chain of data gradients
  int e = run_bwd_begin(c, segs, ptrs);
  for (size_t i = 0; e == PNN_OK && i < segs.size(); ++i) e = run_bwd_body(c, {segs[i]}, {ptrs[i]}, false);
  if (e) return e;
  std::vector<ColRedProb> red;
  e = fire_wgrads(c, segs, ptrs, -1, red);
  if (e) return e;
  return fire_colred(red, c.stream) ? PNN_ERR_HIP : PNN_OK;
}

pnn_status parareal_fine_bwd(pnn_plan* plan, const void* const* dy, const void* const* x,
                             const void* const* phi, const void* saved, void* const* dx, float* const* dphi,
                             void* scratch, void* stream) {
  if (!ok_ctx(plan, const_cast<void*>(saved), scratch)) return PNN_ERR_NULL;
  if (dy == nullptr || x == nullptr || phi == nullptr || dx == nullptr || dphi == nullptr) return PNN_ERR_NULL;
  if (!al_ws(saved, scratch)) return PNN_ERR_ALIGN;
  Ctx c{plan, (char*)const_cast<void*>(saved), (char*)scratch, (hipStream_t)stream};
  std::vector<const SegP*> segs;
  std::vector<Ptrs> ptrs;
  for (int j = 0; j < plan->N; ++j) {
    if (dy[j] == nullptr || x[j] == nullptr || phi[j] == nullptr || dx[j] == nullptr || dphi[j] == nullptr)
      return PNN_ERR_NULL;
    if (!al16({dy[j], x[j], phi[j], dx[j], dphi[j]})) return PNN_ERR_ALIGN;
    Ptrs p;
    p.in = x[j];
    p.params = phi[j];
    p.grads = dphi[j];
    p.gout = dy[j];
    p.gin = dx[j];
    segs.push_back(&plan->fine[j]);
    ptrs.push_back(p);
  }
  return run_bwd_chains(c, segs, ptrs);
}

pnn_status parareal_bwd(pnn_plan* plan, void* const* D, const void* const* rt, const void* const* eta,
                        float* const* deta, const void* const* x, const void* const* phi, void* const* dx,
                        float* const* dphi, const void* saved, void* scratch, void* stream) {
  if (!ok_ctx(plan, const_cast<void*>(saved), scratch)) return PNN_ERR_NULL;
  if (D == nullptr || x == nullptr || phi == nullptr || dx == nullptr || dphi == nullptr) return PNN_ERR_NULL;
  const int N = plan->N;
  if (N > 1 && (rt == nullptr || eta == nullptr || deta == nullptr)) return PNN_ERR_NULL;
  for (int j = 0; j < N; ++j)
    if (D[j] == nullptr || x[j] == nullptr || phi[j] == nullptr || dx[j] == nullptr || dphi[j] == nullptr)
      return PNN_ERR_NULL;
  for (int j = 0; j + 1 < N; ++j) {
    if (rt[j] == nullptr || eta[j] == nullptr || deta[j] == nullptr) return PNN_ERR_NULL;
    if (D[j] == D[j + 1]) return PNN_ERR_SHAPE;
  }
  for (int j = 0; j < N; ++j)
    if (!al16({D[j], x[j], phi[j], dx[j], dphi[j]})) return PNN_ERR_ALIGN;
  for (int j = 0; j + 1 < N; ++j)
    if (!al16({rt[j], eta[j], deta[j]})) return PNN_ERR_ALIGN;
  if (!al_ws(saved, scratch)) return PNN_ERR_ALIGN;
  Ctx c{plan, (char*)const_cast<void*>(saved), (char*)scratch, (hipStream_t)stream};
  std::vector<const SegP*> segs;
  std::vector<Ptrs> ptrs;
  for (int j = 0; j < N; ++j) {
    Ptrs p;
    p.in = x[j];
    p.params = phi[j];
    p.grads = dphi[j];
    p.gout = D[j];
    p.gin = dx[j];
    segs.push_back(&plan->fine[j]);
    ptrs.push_back(p);
  }
  Chains ch;
  int e = chains_group(c, segs, ptrs, ch);
  if (e) return e;
  const int G = (int)ch.ctx.size();
  // the lowest sub-network index of a group: the last D_j of the chain the group needs
  std::vector<int> need(G, N - 1);
  for (int g = 0; g < G; ++g)
    for (auto* sp : ch.segs[g]) need[g] = std::min(need[g], sp->index);
  std::vector<const SegP*> csegs;
  std::vector<Ptrs> cptrs;
  for (int j = N - 2; j >= 0; --j) {
    Ptrs p;
    p.in = rt[j];
    p.params = eta[j];
    p.grads = deta[j];
    p.gout = D[j + 1];
    p.gin = D[j];
    csegs.push_back(&plan->coarse[j]);
    cptrs.push_back(p);
  }
  // Filter transposes depend on the parameters only.  Side streams, after the work enqueued
  // before the call: group 0's (first side stream; the call's stream waits for them after the
  // chain), then each group's own.  The call's stream: every coarse block's in one grouped launch
  // ahead of the chain (group 0's too when there is no side stream).
  e = chains_wait(c, ch, 1, G);
  hipEvent_t t0_done = nullptr;
  if (e == PNN_OK && G > 1) {
    Ctx t0 = ch.ctx[0];
    t0.stream = ch.ctx[1].stream;
    e = run_bwd_begin(t0, ch.segs[0], ch.ptrs[0]);
    t0_done = plan->fj[plan->fj_next++ % plan->fj.size()];
    if (e == PNN_OK && hipEventRecord(t0_done, t0.stream) != hipSuccess) e = PNN_ERR_HIP;
  }
  for (int g = 1; e == PNN_OK && g < G; ++g) e = run_bwd_begin(ch.ctx[g], ch.segs[g], ch.ptrs[g]);
  if (e == PNN_OK) {
    std::vector<const SegP*> ts = csegs;
    std::vector<Ptrs> tp = cptrs;
    if (G == 1) {
      ts.insert(ts.end(), ch.segs[0].begin(), ch.segs[0].end());
      tp.insert(tp.end(), ch.ptrs[0].begin(), ch.ptrs[0].end());
    }
    e = run_bwd_begin(c, ts, tp);
  }
  std::vector<std::vector<ColRedProb>> pending(G);
  // the coarse chain's data gradients on the call's stream; a group starts once its D_j is out
  for (size_t i = 0; e == PNN_OK && i < csegs.size(); ++i) {
    const int j = N - 2 - (int)i;
    e = run_bwd_body(c, {csegs[i]}, {cptrs[i]}, false);
    for (int g = 1; e == PNN_OK && g < G; ++g)
      if (need[g] == j) e = chains_wait(c, ch, g, g + 1);
  }
  // the coarse weight gradients (split-K region 0) wait for the chain on the side stream of the
  // group that starts first, after its own levels; without side streams on the call's stream
  hipEvent_t chain_done = nullptr;
  if (e == PNN_OK && G > 1 && N > 1) {
    chain_done = plan->fj[plan->fj_next++ % plan->fj.size()];
    if (hipEventRecord(chain_done, c.stream) != hipSuccess) e = PNN_ERR_HIP;
  }
  if (e == PNN_OK && t0_done != nullptr && hipStreamWaitEvent(c.stream, t0_done, 0) != hipSuccess) e = PNN_ERR_HIP;
  for (int L = seg_max_level(segs); e == PNN_OK && L >= 1; --L)
    for (int g = 0; e == PNN_OK && g < G; ++g)
      if (L <= seg_max_level(ch.segs[g])) e = run_bwd_level(ch.ctx[g], ch.segs[g], ch.ptrs[g], L, true, pending[g]);
  for (int g = 0; e == PNN_OK && g < G; ++g) e = run_bwd_end(ch.ctx[g], ch.segs[g], ch.ptrs[g], pending[g]);
  if (e == PNN_OK && N > 1) {
    Ctx cw = c;
    if (G > 1) {
      int gw = 1;
      for (int g = 2; g < G; ++g)
        if (need[g] > need[gw]) gw = g;
      cw.stream = ch.ctx[gw].stream;
      if (hipStreamWaitEvent(cw.stream, chain_done, 0) != hipSuccess) e = PNN_ERR_HIP;
    }
    std::vector<ColRedProb> red;
    if (e == PNN_OK) e = fire_wgrads(cw, csegs, cptrs, -1, red);
    if (e == PNN_OK && fire_colred(red, cw.stream)) e = PNN_ERR_HIP;
  }
  const int ej = chains_join(c, ch);
  return e != PNN_OK ? e : ej;
}

pnn_status parareal_combine_bwd(pnn_plan* plan, void* const* dx, const void* const* D, void* stream) {
  if (plan == nullptr) return PNN_ERR_NULL;
  if (plan->N == 1) return PNN_OK;
  if (dx == nullptr || D == nullptr) return PNN_ERR_NULL;
  std::vector<AxpyProb> pr;
  for (int j = 1; j < plan->N; ++j) {
    if (dx[j] == nullptr || D[j - 1] == nullptr) return PNN_ERR_NULL;
    if (!al16({dx[j], D[j - 1]})) return PNN_ERR_ALIGN;
    AxpyProb p;
    p.a = dx[j];
    p.b = D[j - 1];
    p.out = dx[j];
    p.sq_part = nullptr;
    p.n = plan->fine[j].slots[0].elems;
    pr.push_back(p);
  }
  hipStream_t s = (hipStream_t)stream;
  return grouped<AxpyLaunch>(
      pr, [](const AxpyProb& p) { return (int)cdiv(p.n, SUB_TILE); },
      [&](const AxpyLaunch& L, int tiles, size_t) { return launch_sub(L, tiles, plan->dtype, s); });
}

pnn_status pnn_pre_bwd(pnn_plan* plan, const void* image, const void* const* g, const void* const* delta,
                       const void* saved, float* const* ddelta, void* scratch, void* stream) {
  if (!ok_ctx(plan, const_cast<void*>(saved), scratch) || image == nullptr || g == nullptr) return PNN_ERR_NULL;
  if (!al_ws(saved, scratch)) return PNN_ERR_ALIGN;
  Ctx c{plan, (char*)const_cast<void*>(saved), (char*)scratch, (hipStream_t)stream};
  std::vector<const SegP*> segs;
  std::vector<Ptrs> ptrs;
  for (int j = 0; j < plan->N; ++j) {
    const SegP& S = plan->pre[j];
    if (S.grad_bytes == 0 || ddelta == nullptr || ddelta[j] == nullptr) continue;
    if (g[j] == nullptr || delta == nullptr || delta[j] == nullptr) return PNN_ERR_NULL;
    if (!al16({image, g[j], delta[j], ddelta[j]})) return PNN_ERR_ALIGN;
    Ptrs p;
    p.in = image;
    p.params = delta[j];
    p.grads = ddelta[j];
    p.gout = g[j];
    p.gin = nullptr;
    segs.push_back(&S);
    ptrs.push_back(p);
  }
  if (segs.empty()) return PNN_OK;
  // Without BN instances and data gradients (max pools and a convolution on the image) the
  // backward is only the weight gradients, which do not depend on each other: every level in one
  // grouped launch and one column reduce
  bool wgrad_only = true;
  for (auto* sp : segs) {
    if (!sp->bns.empty()) wgrad_only = false;
    for (const NodeP& n : sp->nodes)
      if (n.op == PNN_OP_BNACT || (n.op == PNN_OP_CONV && (n.dgrad || n.dst != sp->out))) wgrad_only = false;
  }
  if (!wgrad_only) return run_bwd(c, segs, ptrs);
  std::vector<ColRedProb> red;
  const int e = fire_wgrads(c, segs, ptrs, -1, red);
  if (e) return e;
  return fire_colred(red, c.stream) ? PNN_ERR_HIP : PNN_OK;
}

pnn_status pnn_inspect(const pnn_plan* plan, int part, int j, int what, int idx, size_t* offset) {
  if (plan == nullptr || offset == nullptr) return PNN_ERR_NULL;
  if (what == 4) {                 // the resident kernel's barrier words (scratch)
    *offset = plan->unit_off;
    return PNN_OK;
  }
  if (what == 5) {                 // the non-finite flags (scratch)
    *offset = plan->flags_off;
    return PNN_OK;
  }
  const std::vector<SegP>* v = part == 0 ? &plan->pre : part == 1 ? &plan->fine : part == 2 ? &plan->coarse : nullptr;
  if (v == nullptr || j < 0 || j >= (int)v->size()) return PNN_ERR_INDEX;
  const SegP& S = (*v)[j];
  if (what == 0 || what == 1) {
    if (idx <= 0 || idx >= (int)S.slots.size() || idx == S.out) return PNN_ERR_INDEX;
    if (what == 0) {
      *offset = S.saved_base + S.slots[idx].saved_off;
      return PNN_OK;
    }
    int s = idx;
    while (S.slots[s].g_off == NONE) {          // residual-only slot: gradient of its consumer
      if (S.slots[s].res_consumer < 0 || !S.needs[s]) return PNN_ERR_INDEX;
      s = S.nodes[S.slots[s].res_consumer].dst;
      if (s == S.out) return PNN_ERR_INDEX;
    }
    *offset = S.scr_base + S.slots[s].g_off;
    return PNN_OK;
  }
  if (idx < 0 || idx >= (int)S.bns.size()) return PNN_ERR_INDEX;
  if (what == 2) {
    if (S.bns[idx].dbn_off == NONE) return PNN_ERR_INDEX;
    *offset = S.scr_base + S.bns[idx].dbn_off;
    return PNN_OK;
  }
  if (what == 3) {
    *offset = S.saved_base + S.bns[idx].stats_off;
    return PNN_OK;
  }
  return PNN_ERR_INDEX;
}

pnn_status pnn_set_streams(pnn_plan* plan, int streams) {
  if (plan == nullptr) return PNN_ERR_NULL;
  if (streams < 1 || streams > PNN_MAX_CHAINS) return PNN_ERR_INDEX;
  // the side streams and the fork / join events, created once (kept for the plan's lifetime)
  while (plan->side.size() + 1 < (size_t)streams) {
    hipStream_t st;
    if (hipStreamCreateWithFlags(&st, hipStreamNonBlocking) != hipSuccess) return PNN_ERR_HIP;
    plan->side.push_back(st);
  }
  while (streams > 1 && plan->fj.size() < 16) {
    hipEvent_t e;
    if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return PNN_ERR_HIP;
    plan->fj.push_back(e);
  }
  plan->streams = streams;
  return PNN_OK;
}

pnn_status pnn_flags_clear(pnn_plan* plan, void* scratch, void* stream) {
  if (plan == nullptr || scratch == nullptr) return PNN_ERR_NULL;
  if (!al(scratch, 256)) return PNN_ERR_ALIGN;
  return launch_flags_clear((unsigned*)((char*)scratch + plan->flags_off), (hipStream_t)stream) ? PNN_ERR_HIP
                                                                                               : PNN_OK;
}

pnn_status pnn_set_resident(pnn_plan* plan, int on) {
  if (plan == nullptr) return PNN_ERR_NULL;
  plan->resident_on = on != 0;
  if (plan->resident_on && plan->unit_cap < 0) plan->unit_cap = unit_fwd_occupancy();
  return PNN_OK;
}

pnn_status pnn_timing_enable(pnn_plan* plan, int family) {
  if (plan == nullptr) return PNN_ERR_NULL;
  if (family < 0 || family > 3) return PNN_ERR_INDEX;
  plan->timing_family = family;
  if (family != 0 && plan->ev.empty()) {
    plan->ev.resize(16384);
    for (auto& e : plan->ev)
      if (hipEventCreate(&e) != hipSuccess) return PNN_ERR_HIP;
  }
  plan->ev_used = 0;
  plan->t_flops = plan->t_bytes = 0.0;
  plan->t_launches = 0;
  return PNN_OK;
}

pnn_status pnn_timing_read(pnn_plan* plan, double* ms, long long* launches, double* flops, double* bytes) {
  if (plan == nullptr || ms == nullptr) return PNN_ERR_NULL;
  double tot = 0.0;
  for (size_t i = 0; i + 1 < plan->ev_used; i += 2) {
    if (hipEventSynchronize(plan->ev[i + 1]) != hipSuccess) return PNN_ERR_HIP;
    float t = 0.f;
    if (hipEventElapsedTime(&t, plan->ev[i], plan->ev[i + 1]) != hipSuccess) return PNN_ERR_HIP;
    tot += t;
  }
  *ms = tot;
  if (launches) *launches = plan->t_launches;
  if (flops) *flops = plan->t_flops;
  if (bytes) *bytes = plan->t_bytes;
  plan->ev_used = 0;
  plan->t_flops = plan->t_bytes = 0.0;
  plan->t_launches = 0;
  return PNN_OK;
}

}  // extern "C"
