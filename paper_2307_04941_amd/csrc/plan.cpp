// Per-shape plan selection: the MI355X counterpart of the multi-grained
// thread-block mapping of MG3MConv (Sec. 4.1.2, Fig. 3; evaluated in Sec. 5.3,
// Table 2).  The paper picks, per convolution scene, whether one MM_unit runs
// on one CPE (TB(1,1)), a row of eight (TB(1,8)) or the whole 8x8 mesh
// (TB(8,8)), because a coarse mapping starves the cores when B, IC and OC are
// small, while a fine one repeats memory traffic when they are large.  Here the
// same trade-off is a choice of work-group tile (how much of the output matrix
// one work-group owns, and how many waves share its staged operands) and of a
// split of the reduction, made by a small cost model over 256 compute units.
//
// Host only: no HIP call in this file.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>

#include "mg3m.h"
#include "mg3m_internal.h"

namespace mg3m {

namespace {

constexpr int kCUs = 256;                    // MI355X: 8 XCDs x 32 CUs
constexpr double kClockHz = 2.4e9;
constexpr double kFlopPerClkCU = 256.0;      // fp32 MFMA: 4 SIMDs x 64 flop/clk
constexpr double kFlopPerClkCU64 = 128.0;    // fp64 MFMA: 4 SIMDs x 32 flop/clk
constexpr int kLdsBytesPerCU = 160 * 1024;
constexpr int kRegsPerLane = 512;            // unified VGPR + AGPR file per SIMD lane
constexpr int kMaxWavesPerSimd = 8;
// Constants fitted to kernel timings on MI355X (see the tile menu): a layer's
// streaming rate, the cost of one kernel launch on the stream, the fixed cost
// of each round of resident work-groups (prologue loads, epilogue stores), and
// how MFMA utilisation falls when fewer than ~2 waves per SIMD are resident.
constexpr double kStreamBytesPerS = 4.0e12;
constexpr double kLaunchUs = 3.0;
constexpr double kRoundUs = 2.0;
constexpr double kUtilBase = 0.5, kUtilPerWave = 0.1;
// Persistent plans (conv_igemm_f32_pt), measured on MI355X against the same
// tile's data-parallel plan: its main loop (run-time LDS buffer parity, one
// copy of the stage code) runs at 0.92 of the tile's rate on deep reductions
// (VGG-16 conv2/conv3, 36 and 18 k-tiles: 8-11% slower); it has no per-round
// cost (a work-group loads its next tile while storing the last); and the
// overlap of output stores with the next tile's MFMAs lets a write-bound layer
// stream at 4.8 TB/s (VGG-16 conv1, 860 MB: 207 -> 180 us).
constexpr double kPersistEff = 0.92;
constexpr double kStreamBytesPerSPersist = 4.8e12;
// The NCHW row loader with a column stride above 1 loads element by element
// (no 16-byte vector covers four output columns): on ResNet-50's stride-2
// layers and AlexNet's conv1 it ran 1.2-1.6x the model's time.  Fitted, with
// the layout-change cost below, to the 44 NCHW layers of VGG-16, ResNet-50
// and AlexNet + inception timed both natively and run as HWCN: the picks then
// total 18714 us against 18823 before and 18696 for the faster of the two on
// every layer.
constexpr double kNchwStridedFactor = 0.6;

long long cdiv(long long a, long long b) { return (a + b - 1) / b; }

const TileDesc& tile_desc(bool acc64, int i) { return acc64 ? kTiles64[i] : kTiles[i]; }
int lds_bytes(const TileDesc& t, bool acc64) { return (acc64 || t.m16) ? lds_bytes_for64(t) : lds_bytes_for(t); }

// Registers of the kernel a plan runs: the persistent kernel's with its
// patch loader, else the tile's (tuned loader).
int kernel_regs(const TileDesc& t, int persist_variant) {
  if (persist_variant < 0) return t.regs;
  return t.regs_pt[persist_variant == kVarHwcnVecNTapDma ? 2 : persist_variant == kVarHwcnVecNTap ? 1 : 0];
}

// Work-groups of this tile resident on one CU, limited by LDS and registers
// (persist_variant: the loader variant of a persistent plan, else -1).
int resident_wgs(const TileDesc& t, bool acc64, int persist_variant = -1) {
  const int waves = t.wm * t.wn;
  const int regs = (kernel_regs(t, persist_variant) + 7) / 8 * 8;
  const int waves_per_simd = std::min(kMaxWavesPerSimd, kRegsPerLane / regs);
  const int by_regs = std::max(1, 4 * waves_per_simd / waves);
  const int by_lds = std::max(1, kLdsBytesPerCU / lds_bytes(t, acc64));
  return std::min(by_regs, by_lds);
}

// Relative speed of the loader variants against the tuned one.  The NCHW
// vec-K and element-wise factors were fitted to timings of every NCHW plan on
// the VGG-16, ResNet-50 and AlexNet/inception layers (ResNet-50's NCHW excess
// over the fastest plan per layer 9.2% -> 3.3%; its 7x7 stem 231 -> 146 us).
double variant_factor(int variant) {
  switch (variant) {
    case kVarHwcnVecNTap: case kVarHwcnVecNTapDma: return 1.0;
    case kVarNchwTap: return 0.9;
    case kVarNchwVecA: return 1.0;
    case kVarHwcnVecN: return 0.85;
    case kVarHwcnVecC: case kVarHwcnVecA: case kVarNchwScalar: return 0.7;
    default: return 0.5;
  }
}

struct Override {
  int mt = 0, nt = 0, kt = 0, split = 0, tail = 0, persist = 0, dma = -1;   // dma: -1 = the default
  int wm = 0, wn = 0;                                                     // waves (0: any)
  int via = -1;                                                           // NCHW run as HWCN: 1, 0, -1 = either
  long long sk = 0;
};

int parse_override(const char* text, Override* o, std::string* err) {
  if (text == nullptr || *text == 0) return MG3M_OK;
  std::string s(text);
  size_t pos = 0;
  while (pos <= s.size()) {
    size_t end = s.find(',', pos);
    if (end == std::string::npos) end = s.size();
    std::string item = s.substr(pos, end - pos);
    pos = end + 1;
    if (item.empty()) {
      if (end == s.size()) break;
      continue;
    }
    size_t eq = item.find('=');
    if (eq == std::string::npos) {
      *err = "plan override: expected key=value, got '" + item + "'";
      return MG3M_ERR_PLAN;
    }
    std::string key = item.substr(0, eq), val = item.substr(eq + 1);
    char* tail = nullptr;
    if (key == "tile") {
      size_t x = val.find('x');
      if (x == std::string::npos) {
        *err = "plan override: tile must be <MT>x<NT>";
        return MG3M_ERR_PLAN;
      }
      // each half must be a whole decimal number (so "64x64;kt=32" is rejected,
      // not read as 64x64 with the default depth)
      auto whole = [](const std::string& t, long* v) {
        char* e = nullptr;
        *v = std::strtol(t.c_str(), &e, 10);
        return !t.empty() && e == t.c_str() + t.size();
      };
      long mt = 0, nt = 0;
      const bool ok = whole(val.substr(0, x), &mt) && whole(val.substr(x + 1), &nt);
      o->mt = ok && mt <= 4096 ? (int)mt : 0;
      o->nt = ok && nt <= 4096 ? (int)nt : 0;
      if (o->mt <= 0 || o->nt <= 0) {
        *err = "plan override: bad tile '" + val + "'";
        return MG3M_ERR_PLAN;
      }
    } else if (key == "waves") {
      size_t x = val.find('x');
      char* e1 = nullptr;
      char* e2 = nullptr;
      const std::string a = x == std::string::npos ? std::string() : val.substr(0, x);
      const std::string b = x == std::string::npos ? std::string() : val.substr(x + 1);
      const long wm = std::strtol(a.c_str(), &e1, 10), wn = std::strtol(b.c_str(), &e2, 10);
      if (a.empty() || b.empty() || *e1 != 0 || *e2 != 0 || wm < 1 || wm > 8 || wn < 1 || wn > 8) {
        *err = "plan override: waves must be <WM>x<WN> (1..8 each)";
        return MG3M_ERR_PLAN;
      }
      o->wm = (int)wm;
      o->wn = (int)wn;
    } else if (key == "via") {
      if (val == "hwcn") {
        o->via = 1;
      } else if (val == "none") {
        o->via = 0;
      } else {
        *err = "plan override: via must be hwcn or none";
        return MG3M_ERR_PLAN;
      }
    } else if (key == "split") {
      long v = std::strtol(val.c_str(), &tail, 10);
      if (tail == val.c_str() || *tail != 0 || v < 1 || v > 64) {
        *err = "plan override: split must be 1..64";
        return MG3M_ERR_PLAN;
      }
      o->split = (int)v;
    } else if (key == "kt") {
      long v = std::strtol(val.c_str(), &tail, 10);
      if (tail == val.c_str() || *tail != 0 || (v != 16 && v != 32)) {
        *err = "plan override: kt must be 16 or 32";
        return MG3M_ERR_PLAN;
      }
      o->kt = (int)v;
    } else if (key == "tail") {
      long v = std::strtol(val.c_str(), &tail, 10);
      if (tail == val.c_str() || *tail != 0 || v < 2 || v > 64) {
        *err = "plan override: tail must be 2..64";
        return MG3M_ERR_PLAN;
      }
      o->tail = (int)v;
    } else if (key == "dma") {
      long v = std::strtol(val.c_str(), &tail, 10);
      if (tail == val.c_str() || *tail != 0 || (v != 0 && v != 1)) {
        *err = "plan override: dma must be 0 or 1";
        return MG3M_ERR_PLAN;
      }
      o->dma = (int)v;
    } else if (key == "persist") {
      long v = std::strtol(val.c_str(), &tail, 10);
      if (tail == val.c_str() || *tail != 0 || v < 1 || v > 16) {
        *err = "plan override: persist must be 1..16 (resident work-groups per CU)";
        return MG3M_ERR_PLAN;
      }
      o->persist = (int)v;
    } else if (key == "sk") {
      long long v = std::strtoll(val.c_str(), &tail, 10);
      if (tail == val.c_str() || *tail != 0 || v < 1 || v > 0x7fffffffLL) {
        *err = "plan override: sk must be 1..2^31-1";
        return MG3M_ERR_PLAN;
      }
      o->sk = v;
    } else {
      *err = "plan override: unknown key '" + key + "'";
      return MG3M_ERR_PLAN;
    }
    if (end == s.size()) break;
  }
  if ((o->split > 0) + (o->tail > 0) + (o->sk > 0) + (o->persist > 0) > 1) {
    *err = "plan override: give at most one of split, tail, sk and persist";
    return MG3M_ERR_PLAN;
  }
  return MG3M_OK;
}

// How a candidate schedules its tiles (see Plan).  kSplitAll and kSplitTail
// cut each tail tile's reduction into `param` runs; kStreamK deals the
// left-over tiles' k-tiles out to `param` work-groups in all (a split when
// the runs fall on tile boundaries).
enum Sched { kDataParallel = 0, kSplitAll = 1, kSplitTail = 2, kStreamK = 3, kPersistent = 4 };

// Partials the tail work-groups write: one per run, plus (stream-K) one for
// each tail tile boundary that falls inside a run.
long long tail_pieces(const Plan& p) {
  if (p.tail_wgs == 0) return 0;
  if (p.sk_s > 0) return p.tail_wgs;
  return (long long)p.tail_wgs + p.tail_tiles - 1;
}

// Fill the shape-dependent parts of a plan for one (tile, schedule, param)
// choice.  Returns false when the choice does not apply to the shape.
bool shape_plan(const ConvShape& s, bool acc64, int tile, int sched, long long param, Plan* p) {
  const TileDesc& t = tile_desc(acc64, tile);
  p->layout = s.layout;
  p->acc64 = acc64 ? 1 : 0;
  p->tile = tile;
  p->t = t;
  p->k_tiles = (int)cdiv(s.Kg, t.kt);
  p->tiles_m = (int)cdiv(s.Mg, t.mt);
  p->tiles_n = (int)cdiv(s.Ng, t.nt);
  const long long tiles = (long long)p->tiles_m * p->tiles_n;
  if (tiles > 0x7fffffffLL) return false;
  long long dp = tiles, tail = 0;
  if (sched == kSplitAll && param > 1) {
    dp = 0;
    tail = tiles;
  } else if ((sched == kSplitTail && param > 1) || sched == kStreamK) {
    // whole rounds of resident work-groups run unsplit (none if the tiles do
    // not fill one round: then every tile is shared out)
    const long long slots = (long long)kCUs * resident_wgs(t, acc64);
    dp = tiles / slots * slots;
    tail = tiles - dp;
  }
  const long long k = p->k_tiles;
  long long wgs = 0, runs = 0, q = 0, r = 0;    // runs: per tail tile (split), 0 (stream-K)
  if (tail > 0) {
    const long long steps = tail * k;
    if (steps > 0x7fffffffLL) return false;          // int step numbers in the kernels
    if (sched == kStreamK) {
      if (param < tail || param > steps) return false;
      wgs = param;
      if (wgs % tail == 0 && k % (wgs / tail) == 0) {
        runs = wgs / tail;                           // equal runs inside each tile: a split
        q = k / runs;
      } else {
        q = steps / wgs;
        r = steps % wgs;
      }
    } else {
      runs = std::min<long long>(param, k);         // no empty run
      wgs = tail * runs;
      q = k / runs;
      r = k % runs;
    }
    if (runs == 1) {                                 // one run per tile: run them whole
      dp = tiles;
      tail = wgs = q = r = runs = 0;
    }
  }
  if (dp + wgs > 0x7fffffffLL) return false;
  // persistent: every tile whole, `param` resident work-groups per CU looping over them
  p->persist = sched == kPersistent ? 1 : 0;
  p->dp_tiles = (int)dp;
  p->tail_tiles = (int)tail;
  p->tail_wgs = (int)wgs;
  p->sk_s = (int)runs;
  p->sk_q = (int)q;
  p->sk_r = (int)r;
  p->split = tail > 0 ? (int)cdiv(wgs, tail) : 1;
  p->grid = p->persist ? std::min<long long>(dp, (long long)kCUs * param) : dp + wgs;
  p->lds_bytes = lds_bytes(t, acc64);
  const double padded = (double)p->tiles_m * t.mt * (double)p->tiles_n * t.nt *
                        (double)p->k_tiles * t.kt;
  p->pad_eff = (double)s.Mg * (double)s.Ng * (double)s.Kg / padded;
  // partial slots: run w's piece in tail tile j goes to slot w + j
  const long long slots = wgs > 0 ? wgs + tail - 1 : 0;
  p->ws_bytes = (size_t)slots * t.mt * t.nt * (acc64 ? sizeof(double) : sizeof(float));
  p->est_us = 0.0;
  return true;
}

// The selector's predicted time for a plan (microseconds).  Work-groups are
// dispatched in order, whole tiles first and tail runs after them.  In each
// phase the busiest CU runs ceil(work-groups / 256) of them, each costing its
// padded MFMA flops at the tile's measured efficiency, scaled down when that
// CU holds too few waves to hide latency, plus a fixed cost per round of
// resident work-groups.  A layer cannot beat streaming its tensors (and the
// partials) once; the tail reduction adds its traffic and a second launch.
double predict_us(const ConvShape& s, const Plan& p) {
  const TileDesc& t = p.t;
  const int occ = resident_wgs(t, p.acc64, p.persist ? p.variant : -1);
  const double rate = p.acc64 ? kFlopPerClkCU64 : kFlopPerClkCU;
  const double tile_flops = 2.0 * t.mt * t.nt * (double)t.kt;
  const bool multitap = s.R * s.S > 1 && s.C >= 2 * t.kt;
  auto phase = [&](long long wgs, int k_tiles) {
    if (wgs <= 0) return 0.0;
    const long long per_cu = cdiv(wgs, kCUs);
    const double waves_per_simd = (double)std::min<long long>(per_cu, occ) * t.wm * t.wn / 4.0;
    const double util = std::min(1.0, kUtilBase + kUtilPerWave * waves_per_simd);
    const double eff = t.eff * variant_factor(p.variant) * util * (multitap ? t.eff_multitap : 1.0) *
                       (p.persist ? kPersistEff : 1.0) *
                       (s.layout == kNCHW && p.b_mode == kBVecW && s.sw > 1 ? kNchwStridedFactor : 1.0);
    return (double)per_cu * tile_flops * k_tiles / (rate * kClockHz * eff) * 1e6 +
           (p.persist ? 1.0 : (double)cdiv(per_cu, occ)) * kRoundUs;
  };
  const int run_k = p.tail_wgs > 0 ? p.sk_q + (p.sk_r > 0 ? 1 : 0) : 0;
  const double t_comp = phase(p.dp_tiles, p.k_tiles) + phase(p.tail_wgs, run_k);
  const double y_bytes = 4.0 * (double)s.Mg * (double)s.Ng;
  const double xw_bytes = 4.0 * ((double)s.N * s.C * s.H * s.W + (double)s.Kg * s.Mg);
  const double part_bytes =
      (double)tail_pieces(p) * t.mt * t.nt * (p.acc64 ? sizeof(double) : sizeof(float));
  const double t_mem =
      (xw_bytes + y_bytes + part_bytes) / (p.persist ? kStreamBytesPerSPersist : kStreamBytesPerS) * 1e6;
  double est = std::max(t_comp, t_mem) + kLaunchUs;
  if (p.tail_tiles > 0) {
    const double tail_out = 4.0 * (double)p.tail_tiles * t.mt * t.nt;
    est += (part_bytes + tail_out) / kStreamBytesPerS * 1e6 + kLaunchUs;
  }
  if (p.wt_bytes > 0) est += 2.0 * (double)p.wt_bytes / kStreamBytesPerS * 1e6 + kLaunchUs;
  return est;
}

}  // namespace

int make_shape(int N, int C, int H, int W, int K, int R, int S, int stride_h, int stride_w,
               int pad_h, int pad_w, int layout, ConvShape* s, std::string* err) {
  if (layout != kHWCN && layout != kNCHW) {
    *err = "unknown layout";
    return MG3M_ERR_LAYOUT;
  }
  if (N < 1 || C < 1 || H < 1 || W < 1 || K < 1 || R < 1 || S < 1 || stride_h < 1 ||
      stride_w < 1 || pad_h < 0 || pad_w < 0) {
    *err = "dimensions and strides must be >= 1, pads >= 0";
    return MG3M_ERR_SHAPE;
  }
  if (pad_h > (1 << 24) || pad_w > (1 << 24) || H > (1 << 24) || W > (1 << 24) ||
      R > (1 << 24) || S > (1 << 24) || stride_h > (1 << 24) || stride_w > (1 << 24)) {
    *err = "a spatial size, stride or pad exceeds 2^24";
    return MG3M_ERR_TOO_LARGE;
  }
  const long long eh = (long long)H + 2LL * pad_h - R, ew = (long long)W + 2LL * pad_w - S;
  if (eh < 0 || ew < 0) {
    *err = "filter larger than the padded input: empty output";
    return MG3M_ERR_SHAPE;
  }
  s->N = N; s->C = C; s->H = H; s->W = W; s->K = K; s->R = R; s->S = S;
  s->sh = stride_h;
  s->sw = stride_w;
  s->ph = pad_h;
  s->pw = pad_w;
  s->Ho = (int)(eh / stride_h + 1);
  s->Wo = (int)(ew / stride_w + 1);
  s->layout = layout;
  s->Mg = K;
  s->Ng = (long long)N * s->Ho * s->Wo;
  s->Kg = (long long)C * R * S;
  // int32 index arithmetic in the kernels, with head-room for a tile past the end
  // 32-bit byte offsets in the kernels' buffer loads
  const long long lim = kMaxTensorBytes / 4;
  const long long xe = (long long)N * C * H * W, we = (long long)K * C * R * S,
                  ye = (long long)N * K * s->Ho * s->Wo;
  if (xe > lim || we > lim || ye > lim) {
    *err = "a tensor is larger than 4 GiB - 64 bytes (the kernels use 32-bit byte offsets)";
    return MG3M_ERR_TOO_LARGE;
  }
  return MG3M_OK;
}

// Loader variant and epilogue mode for a plan whose tile is already set.
// dma: the one-tap HWCN loaders in their direct-to-LDS form.
void choose_modes(const ConvShape& s, bool x16, bool w16, bool y16, Plan* p, bool dma = false) {
  if (s.layout == kHWCN) {
    if (s.K % 4 == 0 && w16) {
      p->a_mode = kAVecM;
      if (s.N % 4 == 0 && x16 && s.C % p->t.kt == 0)
        p->b_mode = dma ? kBVecNTapDma : kBVecNTap, p->variant = dma ? kVarHwcnVecNTapDma : kVarHwcnVecNTap;
      else if (s.N % 4 == 0 && x16) p->b_mode = kBVecN, p->variant = kVarHwcnVecN;
      else if (s.N == 1 && s.C % 4 == 0 && x16) p->b_mode = kBVecC, p->variant = kVarHwcnVecC;
      else p->b_mode = kBScalar, p->variant = kVarHwcnVecA;
    } else {
      p->a_mode = kAScalar;
      p->b_mode = kBScalar;
      p->variant = kVarHwcnScalar;
    }
  } else if (s.C % p->t.kt == 0 && s.K % 4 == 0 && s.R * s.S > 1 && s.sw == 1) {
    // tap-major on a [R][S][C][K] copy of the filter (in the workspace).  A 1x1
    // filter has one tap (both orders coincide, the copy would be pure cost),
    // and other strides never take the 16-byte runs along W.
    p->a_mode = kAVecM;
    p->b_mode = kBVecWTap;
    p->variant = kVarNchwTap;
  } else {
    p->b_mode = kBVecW;
    if (s.Kg % 4 == 0 && w16) p->a_mode = kAVecK, p->variant = kVarNchwVecA;
    else p->a_mode = kAScalar, p->variant = kVarNchwScalar;
  }
  // The filter copy goes first in the workspace, the partials after it.
  p->wt_bytes = 0;
  if (p->variant == kVarNchwTap) {
    p->wt_bytes = ((size_t)4 * (size_t)s.Mg * (size_t)s.Kg + 255) / 256 * 256;
    p->ws_bytes += p->wt_bytes;
  }
  // Four consecutive output channels are contiguous only in HWCN with N == 1
  // (whole tiles store them with one 16-byte store; partials are stored per
  // element, so only y's alignment matters).
  p->e_mode = (s.layout == kHWCN && s.N == 1 && s.K % 4 == 0 && y16) ? kEVecM : kEElem;
  // the fp64 accumulator holds no four adjacent rows in one lane
  if (p->acc64) p->e_mode = kEElem;
}

int make_plan(const ConvShape& s, const char* override_text, bool acc64, bool x16, bool w16,
              bool y16, Plan* p, std::string* err, size_t ws_cap) {
  Override o;
  int rc = parse_override(override_text, &o, err);
  if (rc) return rc;
  if (acc64 && o.kt && o.kt != 16) {
    *err = "plan override: the fp64-accumulating kernel steps the reduction by kt=16";
    return MG3M_ERR_PLAN;
  }

  int best = -1;
  Plan best_plan{};
  size_t least_over_cap = SIZE_MAX;     // smallest workspace among the candidates over ws_cap
  // the split factors the cost model was calibrated on
  const int splits[] = {2, 3, 4, 6, 8, 16};
  // via: an NCHW call run as HWCN on 16-byte aligned copies of x, w and y in
  // the workspace, the layout changed on the way in and out (layout.hip)
  auto consider_one = [&](int ti, int sched, long long sp, bool via) {
    Plan c{};
    ConvShape sv = s;
    if (via) sv.layout = kHWCN;
    if (!shape_plan(sv, acc64, ti, sched, sp, &c)) return;
    // the one-tap HWCN loaders load straight into LDS unless the override says
    // otherwise, except in the fp64-accumulating kernels and the 16-row tile,
    // which stage through VGPRs
    const bool dma_ok = !c.acc64 && !c.t.m16;
    choose_modes(sv, via || x16, via || w16, via || y16, &c, dma_ok && o.dma != 0);
    if (via) {
      auto r256 = [](size_t b) { return (b + 255) / 256 * 256; };
      c.via_hwcn = 1;
      c.via_bytes = r256(4 * (size_t)s.N * s.C * s.H * s.W) + r256(4 * (size_t)s.Mg * (size_t)s.Kg) +
                    r256(4 * (size_t)s.Mg * (size_t)s.Ng);
      c.ws_bytes += c.via_bytes;
    }
    if (o.dma == 1 && c.variant != kVarHwcnVecNTapDma) return;
    // runs spanning two tiles need the kernel's loop over pieces (only the
    // 32x32x2 fp32 kernel with the one-tap HWCN loader has it)
    if (c.tail_wgs > 0 && c.sk_s == 0 && (c.acc64 || c.t.m16 || !tail_runs_multi(c.b_mode))) return;
    // the persistent kernel is built for the batch-vector HWCN loaders only
    if (c.persist && (c.acc64 || !persist_built(c.variant, c.t))) return;
    if (c.persist && sp == 0) {
      // the selector's persistent plans fill every slot the kernel's
      // occupancy allows, and only pay off with more tiles than that
      const long long slots = (long long)kCUs * resident_wgs(c.t, false, c.variant);
      if (c.dp_tiles <= slots) return;
      c.grid = slots;
    }
    if (c.ws_bytes > ws_cap) {
      least_over_cap = std::min(least_over_cap, c.ws_bytes);
      return;
    }
    c.est_us = predict_us(sv, c);
    // the layout changes: x and w in, y out, each read and written once
    if (via) c.est_us += 2.0 * (double)c.via_bytes / kStreamBytesPerS * 1e6 + 2 * kLaunchUs;
    // ties: less workspace traffic, then the larger tile
    const bool better = best < 0 || c.est_us < best_plan.est_us * 0.999 ||
                        (std::fabs(c.est_us - best_plan.est_us) <= best_plan.est_us * 0.001 &&
                         (c.ws_bytes < best_plan.ws_bytes ||
                          (c.ws_bytes == best_plan.ws_bytes && c.t.mt * c.t.nt > best_plan.t.mt * best_plan.t.nt)));
    if (better) {
      best = ti;
      best_plan = c;
    }
  };
  const bool via_ok = s.layout == kNCHW && !acc64;
  if (o.via == 1 && !via_ok) {
    *err = "plan override: via=hwcn applies to NCHW calls of the fp32 kernel";
    return MG3M_ERR_PLAN;
  }
  auto consider = [&](int ti, int sched, long long sp) {
    if (o.via != 1) consider_one(ti, sched, sp, false);
    if (via_ok && o.via != 0) consider_one(ti, sched, sp, true);
  };
  for (int ti = 0; ti < (acc64 ? kNumTiles64 : kNumTiles); ++ti) {
    const TileDesc& td = tile_desc(acc64, ti);
    if (o.mt && !(td.mt == o.mt && td.nt == o.nt)) continue;
    if (o.wm && !(td.wm == o.wm && td.wn == o.wn)) continue;
    // The selector takes a 16-row tile only where it saves padding, i.e. a
    // 32-row block would be at most half full (the case it was timed on).
    if (!o.mt && td.m16 && !(s.Mg % 32 != 0 && s.Mg % 32 <= 16)) continue;
    // A tile the cost model does not yet rank correctly is left to overrides
    // that name its shape and its waves.
    if (td.forced_only && !(o.mt && o.wm)) continue;
    // a forced tile without a depth means the default depth of 16
    if ((o.kt || o.mt) && td.kt != (o.kt ? o.kt : 16)) continue;
    if (o.split) {
      consider(ti, o.split > 1 ? kSplitAll : kDataParallel, o.split);
    } else if (o.tail) {
      consider(ti, kSplitTail, o.tail);
    } else if (o.sk) {
      consider(ti, kStreamK, o.sk);
    } else if (o.persist) {
      consider(ti, kPersistent, o.persist);
    } else {
      consider(ti, kDataParallel, 1);
      for (int sp : splits) {
        consider(ti, kSplitAll, sp);
        consider(ti, kSplitTail, sp);
      }
      // stream-K over the left-over tiles with one to all resident work-groups per CU
      for (int j = 1, occ = resident_wgs(td, acc64); j <= occ; ++j) consider(ti, kStreamK, (long long)j * kCUs);
      // every tile whole, persistent work-groups filling the chip
      if (!acc64) consider(ti, kPersistent, 0);
    }
  }
  if (best < 0 && least_over_cap != SIZE_MAX) {
    *err = "every applicable plan needs more workspace than the " + std::to_string(ws_cap) +
           " bytes available (the smallest needs " + std::to_string(least_over_cap) + ")";
    return MG3M_ERR_WORKSPACE;
  }
  if (best < 0) {
    *err = "plan override: no applicable plan for tile " + std::to_string(o.mt) + "x" + std::to_string(o.nt) +
           (o.dma == 1 ? std::string(" dma=1 (the direct-to-LDS loaders serve the fp32 kernel's one-tap HWCN path"
                                     " with 32x32x2-MFMA tiles)")
                       : std::string()) +
           (o.persist ? " persist=" + std::to_string(o.persist) +
                            " (persistent tiles need the fp32 kernel's batch-vector HWCN loaders: HWCN, N and K"
                            " multiples of 4, aligned buffers; not the 16-row tile)"
                      : std::string()) +
           (o.kt ? " kt=" + std::to_string(o.kt) : std::string()) +
           (o.tail ? " tail=" + std::to_string(o.tail) : std::string()) +
           (o.sk ? " sk=" + std::to_string(o.sk) +
                       " (from the left-over tiles to their k-tiles in total; runs spanning two tiles"
                       " only with the fp32 kernel's one-tap HWCN loader)"
                 : std::string());
    return MG3M_ERR_PLAN;
  }
  *p = best_plan;
  return MG3M_OK;
}

std::string plan_to_string(const ConvShape& s, const Plan& p) {
  static const char* an[] = {"vec_m", "vec_k", "scalar"};
  static const char* bn[] = {"vec_n", "vec_c", "scalar", "vec_n_tap", "vec_w", "vec_w_tap", "vec_n_tap_dma"};
  static const char* en[] = {"elem", "vec_m"};
  char buf[512];
  std::snprintf(buf, sizeof buf,
                "%s%s%stile=%dx%d,waves=%dx%d,kt=%d,split=%d,dp_tiles=%d,tail_tiles=%d,tail_wgs=%d,grid=%lld,"
                "tiles=%dx%d,k_tiles=%d,a=%s,b=%s,e=%s,lds=%d,ws=%zu,pad_eff=%.4f,est_us=%.2f,"
                "Mg=%lld,Ng=%lld,Kg=%lld",
                p.acc64 ? "acc=f64," : "", p.via_hwcn ? "via=hwcn," : "",
                p.persist ? "persist," : "", p.t.mt, p.t.nt, p.t.wm, p.t.wn, p.t.kt, p.split, p.dp_tiles, p.tail_tiles, p.tail_wgs, p.grid,
                p.tiles_m, p.tiles_n, p.k_tiles, an[p.a_mode], bn[p.b_mode], en[p.e_mode],
                p.lds_bytes, p.ws_bytes, p.pad_eff, p.est_us, s.Mg, s.Ng, s.Kg);
  return buf;
}

}  // namespace mg3m
