// Host side of librt3d: argument validation, the compact KGS pack (Section 3
// of RT3D, arXiv 2007.09835: a kernel group reshaped to g_M x (g_N*K_s)
// loses whole columns), the launch planner that lays the kept weights out in
// MFMA operand order, and the C entry points declared in include/rt3d.h.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <map>
#include <mutex>
#include <numeric>
#include <tuple>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "rt3d_internal.h"

namespace rt3d {
namespace {

thread_local std::string g_detail;

rt3d_status fail(rt3d_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_detail = buf;
  return s;
}

rt3d_status ok() {
  g_detail.clear();
  return RT3D_OK;
}

int esize_of(int dtype) { return dtype == RT3D_F32 ? 4 : 2; }

// Benchmark-only overrides of planner choices, all read from one variable,
// RT3D_TUNE="key=value,key=value" (keys and effects are listed in
// include/rt3d.h).  Returns -1 when the key is absent.  Unset in normal use.
int tune(const char *key) {
  const char *env = std::getenv("RT3D_TUNE");
  if (!env) return -1;
  const size_t n = std::strlen(key);
  for (const char *p = env; *p;) {
    while (*p == ',' || *p == ' ') ++p;
    if (std::strncmp(p, key, n) == 0 && p[n] == '=') return std::atoi(p + n + 1);
    while (*p && *p != ',') ++p;
  }
  return -1;
}

uint64_t align_up(uint64_t v, uint64_t a) { return (v + a - 1) / a * a; }

int out_len(int in, int k, int s, int p) {
  const int span = in + 2 * p - k;
  return span < 0 ? 0 : span / s + 1;
}

// ---------------------------------------------------------------------------
// Validation
// ---------------------------------------------------------------------------

rt3d_status check_desc(const rt3d_conv3d_desc *d, bool need_groups) {
  if (!d) return fail(RT3D_ERR_INVALID_ARG, "desc is NULL");
  if (d->n < 0) return fail(RT3D_ERR_INVALID_ARG, "batch n=%d is negative", d->n);
  if (d->c_in <= 0 || d->c_out <= 0 || d->t <= 0 || d->h <= 0 || d->w <= 0)
    return fail(RT3D_ERR_INVALID_ARG, "channel and extent sizes must be positive");
  if (d->kt <= 0 || d->kh <= 0 || d->kw <= 0 || d->st <= 0 || d->sh <= 0 || d->sw <= 0 ||
      d->pt < 0 || d->ph < 0 || d->pw < 0)
    return fail(RT3D_ERR_INVALID_ARG, "kernel extents and strides must be positive, padding >= 0");
  if (d->dtype != RT3D_F32 && d->dtype != RT3D_BF16 && d->dtype != RT3D_F16)
    return fail(RT3D_ERR_INVALID_ARG, "unknown dtype %d", d->dtype);
  if (d->flags & ~(RT3D_RELU | RT3D_RESIDUAL))
    return fail(RT3D_ERR_INVALID_ARG, "unknown flag bits 0x%x", d->flags);
  if (out_len(d->t, d->kt, d->st, d->pt) <= 0 || out_len(d->h, d->kh, d->sh, d->ph) <= 0 ||
      out_len(d->w, d->kw, d->sw, d->pw) <= 0)
    return fail(RT3D_ERR_INVALID_ARG, "the kernel does not fit the padded input");
  if (d->kt > 7 || d->kh > 7 || d->kw > 7)
    return fail(RT3D_ERR_UNSUPPORTED, "kernel extents above 7 are not supported");
  if (d->st > 2 || d->sh > 2 || d->sw > 2)
    return fail(RT3D_ERR_UNSUPPORTED, "strides above 2 are not supported");
  if (d->pt >= d->kt || d->ph >= d->kh || d->pw >= d->kw)
    return fail(RT3D_ERR_UNSUPPORTED, "padding must be smaller than the kernel extent");
  if (d->qt < 0 || d->qh < 0 || d->qw < 0)
    return fail(RT3D_ERR_INVALID_ARG, "pooling windows must be >= 0");
  if (d->qt > 8 || d->qh > 8 || d->qw > 8)
    return fail(RT3D_ERR_UNSUPPORTED, "pooling windows above 8 are not supported");
  {
    const int qt = std::max(1, d->qt), qh = std::max(1, d->qh), qw = std::max(1, d->qw);
    if (out_len(d->t, d->kt, d->st, d->pt) / qt <= 0 || out_len(d->h, d->kh, d->sh, d->ph) / qh <= 0 ||
        out_len(d->w, d->kw, d->sw, d->pw) / qw <= 0)
      return fail(RT3D_ERR_INVALID_ARG, "the pooling window does not fit the conv output");
  }
  if (d->y_c_total != 0 || d->y_c_off != 0) {
    if (d->y_c_off < 0 || d->y_c_total < d->c_out ||
        static_cast<long>(d->y_c_off) + d->c_out > d->y_c_total)
      return fail(RT3D_ERR_INVALID_ARG, "output channels [%d, %d) do not fit y_c_total=%d",
                  d->y_c_off, d->y_c_off + d->c_out, d->y_c_total);
    if (d->y_c_total % 4 != 0 || d->y_c_off % 4 != 0)
      return fail(RT3D_ERR_UNSUPPORTED, "y_c_total and y_c_off must be multiples of 4");
  }
  if (d->x_c_total != 0 || d->x_c_off != 0) {
    if (d->x_c_off < 0 || d->x_c_total < d->c_in ||
        static_cast<long>(d->x_c_off) + d->c_in > d->x_c_total)
      return fail(RT3D_ERR_INVALID_ARG, "input channels [%d, %d) do not fit x_c_total=%d",
                  d->x_c_off, d->x_c_off + d->c_in, d->x_c_total);
    if (d->c_in <= 4 && (d->x_c_total != d->c_in || d->x_c_off != 0))
      return fail(RT3D_ERR_UNSUPPORTED, "layers with c_in <= 4 read whole voxels");
  }
  if (need_groups) {
    auto okg = [](int g) { return g == 4 || g == 8 || g == 16; };
    if (!okg(d->g_m) || !okg(d->g_n))
      return fail(RT3D_ERR_UNSUPPORTED, "group sizes g_m=%d g_n=%d: only 4, 8, 16", d->g_m, d->g_n);
  }
  // 32-bit LDS offsets and step counters bound the layer size.
  const double elems = static_cast<double>(d->c_out) * d->c_in * d->kt * d->kh * d->kw;
  if (elems > 1.0e9) return fail(RT3D_ERR_UNSUPPORTED, "weight tensor too large");
  return ok();
}

uint64_t desc_hash(const rt3d_conv3d_desc *d) {
  const int32_t f[] = {d->c_in, d->c_out, d->t,  d->h,  d->w,   d->kt,    d->kh,
                       d->kw,   d->st,    d->sh, d->sw, d->pt,  d->ph,    d->pw,
                       d->g_m,  d->g_n,   d->dtype, std::max(1, d->qt), std::max(1, d->qh),
                       std::max(1, d->qw)};
  uint64_t h = 1469598103934665603ull;
  for (int32_t v : f) {
    for (int b = 0; b < 4; ++b) {
      h ^= static_cast<uint8_t>(static_cast<uint32_t>(v) >> (8 * b));
      h *= 1099511628211ull;
    }
  }
  return h;
}

// ---------------------------------------------------------------------------
// Layer geometry and the voxel tiling
// ---------------------------------------------------------------------------

struct Geom {
  int n, c_in, c_out, t, h, w, kt, kh, kw, st, sh, sw, pt, ph, pw, to, ho, wo, ks, es;
  int qt, qh, qw, pto, pho, pwo;  // fused pooling window and pooled extent
};

Geom geom_of(const rt3d_conv3d_desc *d) {
  Geom g{d->n,  d->c_in, d->c_out, d->t,  d->h,  d->w,  d->kt, d->kh, d->kw, d->st,
         d->sh, d->sw,   d->pt,    d->ph, d->pw, 0,     0,     0,     0,     0,
         1,     1,       1,        0,     0,     0};
  g.to = out_len(d->t, d->kt, d->st, d->pt);
  g.ho = out_len(d->h, d->kh, d->sh, d->ph);
  g.wo = out_len(d->w, d->kw, d->sw, d->pw);
  g.ks = d->kt * d->kh * d->kw;
  g.es = esize_of(d->dtype);
  g.qt = std::max(1, d->qt);
  g.qh = std::max(1, d->qh);
  g.qw = std::max(1, d->qw);
  g.pto = g.to / g.qt;
  g.pho = g.ho / g.qh;
  g.pwo = g.wo / g.qw;
  return g;
}

constexpr int kSlots = 128;            // voxel slots per workgroup
constexpr int kMaxHalo = 96 * 1024;    // LDS bytes for the staged brick

// Choose the output brick: fewest launched voxel slots (least waste at the
// volume's edges), then the smallest halo (least staging traffic).
Tiling choose_tiling(const Geom &g, int slots = kSlots) {
  Tiling best{};
  long best_cost = -1, best_halo = 0;
  // Channels per LDS chunk: 32 (16-bit) or 16 (fp32), narrower when the
  // layer has fewer input channels (a whole 16-byte piece at least).
  const int epp = 16 / g.es;
  int cc = epp;  // smallest power-of-two multiple of a piece covering c_in, capped
  while (cc < g.c_in && cc < (g.es == 2 ? 32 : 16)) cc *= 2;
  // LDS row pitch: an odd multiple of 16 bytes (4 banks), so that 16 voxels
  // whose halo indices differ modulo 16 start on 16 distinct bank quads and
  // two 8-byte item reads in one pass are conflict-free when their channel
  // blocks differ in parity (see pair_items).
  int row = (cc * g.es + 15) / 16 * 16;
  if ((row / 16) % 2 == 0) row += 16;
  // Bricks hold whole pooling windows (their origins are then multiples of
  // the window too), so the fused pooling never crosses workgroups.
  for (int bw = g.qw; bw <= std::max(g.qw, std::min(g.wo, slots)); bw += g.qw)
    for (int bh = g.qh; bh <= std::max(g.qh, std::min(g.ho, slots / bw)); bh += g.qh)
      for (int bt = g.qt; bt <= std::max(g.qt, std::min(g.to, slots / (bw * bh))); bt += g.qt) {
        if (bt * bh * bw > slots) continue;
        const int ht = (bt - 1) * g.st + g.kt;
        const int hh = (bh - 1) * g.sh + g.kh;
        const int hw = (bw - 1) * g.sw + g.kw;
        const long halo = static_cast<long>(ht) * hh * hw * row;
        if (halo > kMaxHalo) continue;
        const long nb = static_cast<long>((g.to + bt - 1) / bt) * ((g.ho + bh - 1) / bh) *
                        ((g.wo + bw - 1) / bw);
        // LDS bank-conflict degree of a 16-voxel fragment: the largest number
        // of its voxels whose halo row index coincides modulo 16 (modulo 8
        // for the 16-byte fp32 reads).
        const int modulus = g.es == 2 ? 16 : 8;
        int conflict = 1;
        for (int f = 0; f < slots / 16; ++f) {
          int hits[16] = {0};
          for (int n = 0; n < 16; ++n) {
            const int sl = 16 * f + n;
            const int tt = sl / (bh * bw), hh2 = (sl / bw) % bh, ww = sl % bw;
            if (tt >= bt) continue;
            const int v = ((tt * g.st) * hh + hh2 * g.sh) * hw + ww * g.sw;
            conflict = std::max(conflict, ++hits[v % modulus]);
          }
        }
        const long cost = nb * slots * (3 + conflict);
        if (best_cost < 0 || cost < best_cost || (cost == best_cost && halo < best_halo)) {
          best_cost = cost;
          best_halo = halo;
          best = Tiling{bt, bh, bw, ht, hh, hw, cc, row, slots, (g.c_in + cc - 1) / cc};
        }
      }
  // 16-bit layers with a small halo (few kernel taps) take wider channel
  // chunks: each chunk then carries more K-steps per halo load, barrier and
  // pipeline restart.  Limits: the register stager's 8 pieces of 16 bytes
  // per thread (2048 per workgroup) and the LDS budget.  Layers of fewer
  // than 256 output voxels whose narrow chunks already carry 16 or more
  // K-steps keep them: they split their channels across workgroups, and
  // finer chunks balance the splits (C3D conv5a/b at batch 1: 12.6 -> 11.6
  // us KGS, 13.4 -> 12.1 dense; factorised 1x3x3 / 3x1x1 layers of that size
  // ran 1-2 us slower on narrow chunks).
  const long out_vox = static_cast<long>(std::max(g.n, 1)) * g.to * g.ho * g.wo;
  const bool keep_narrow = out_vox < 256 && (best.cc / 4) * g.ks / 8 >= 16;
  if (best_cost >= 0 && g.es == 2 && !keep_narrow) {
    int wide = best.cc;
    const int cap = tune("cc") >= 8 ? tune("cc") : 128;  // tuning switch cc=N caps the width
    while (wide < cap && wide < g.c_in) {
      const int next = wide * 2;
      int nrow = (next * g.es + 15) / 16 * 16;
      if ((nrow / 16) % 2 == 0) nrow += 16;
      const long rows = static_cast<long>(best.ht) * best.hh * best.hw;
      if (rows * (next / 8) > 2048 || rows * nrow > kMaxHalo) break;
      wide = next;
      best.row = nrow;
    }
    best.cc = wide;
    best.nchunks = (g.c_in + wide - 1) / wide;
  }
  return best;
}

// LDS byte offset of the item (channel block ql of the chunk, kernel
// position pos) relative to a voxel slot's (0,0,0) tap.
uint32_t item_offset(const Geom &g, const Tiling &tl, int ql, int pos) {
  const int iw = pos % g.kw;
  const int ih = (pos / g.kw) % g.kh;
  const int it = pos / (g.kw * g.kh);
  return static_cast<uint32_t>(((it * tl.hh + ih) * tl.hw + iw) * tl.row + ql * 4 * g.es);
}

// ---------------------------------------------------------------------------
// Canonical KGS sections (the compact per-group format of Section 3)
// ---------------------------------------------------------------------------

struct Canon {
  int P, Q;
  std::vector<uint32_t> group_ptr;
  std::vector<uint16_t> pos;
  std::vector<uint64_t> val_ptr;
  uint64_t nvals = 0;
};

rt3d_status canon_index(const rt3d_conv3d_desc *d, const uint8_t *mask, Canon &c) {
  const int ks = d->kt * d->kh * d->kw;
  c.P = (d->c_out + d->g_m - 1) / d->g_m;
  c.Q = (d->c_in + d->g_n - 1) / d->g_n;
  c.group_ptr.assign(static_cast<size_t>(c.P) * c.Q + 1, 0);
  c.val_ptr.assign(static_cast<size_t>(c.P) * c.Q + 1, 0);
  c.pos.clear();
  uint64_t nv = 0;
  for (int p = 0; p < c.P; ++p) {
    const int gm = std::min(d->g_m, d->c_out - p * d->g_m);
    for (int q = 0; q < c.Q; ++q) {
      const int gn = std::min(d->g_n, d->c_in - q * d->g_n);
      const size_t gi = static_cast<size_t>(p) * c.Q + q;
      const uint8_t *row = mask + gi * ks;
      c.group_ptr[gi] = static_cast<uint32_t>(c.pos.size());
      c.val_ptr[gi] = nv;
      int k = 0;
      for (int s = 0; s < ks; ++s) {
        if (row[s] > 1)
          return fail(RT3D_ERR_INVALID_ARG, "mask[%d][%d][%d] = %d is not 0 or 1", p, q, s, row[s]);
        if (row[s]) {
          c.pos.push_back(static_cast<uint16_t>(s));
          ++k;
        }
      }
      nv += static_cast<uint64_t>(gm) * gn * k;
    }
  }
  c.group_ptr.back() = static_cast<uint32_t>(c.pos.size());
  c.val_ptr.back() = nv;
  c.nvals = nv;
  return ok();
}

// Small-input-channel path (kVarSmall*16): 16-bit, c_in <= 4 (one 4-channel
// block per tap), a halo of at most 12 lines (kt * (sh + kh)) of at most 253
// elements ((31 sw + kw) * c_in: one 8-byte word per lane, from the aligned
// word at or before the line start), w * c_in % 4 == 0 (every halo line of a
// brick then starts at the same offset within its word), at most 64 taps (8
// K-steps of 8), and pooling that is either absent or 1x2x2 (the brick's two
// rows and adjacent lanes).  The input must also stay below 2^31 - 8 bytes (its buffer
// resource extent), checked at launch.  Tuning switch small_kernel=0 disables it.
bool small_ok(const Geom &g) {
  if (tune("small_kernel") == 0) return false;
  const bool pool_ok = (g.qt == 1 && g.qh == 1 && g.qw == 1) || (g.qt == 1 && g.qh == 2 && g.qw == 2);
  const int lines = g.kt * (g.sh + g.kh);
  const int line_elems = (31 * g.sw + g.kw) * g.c_in;
  return g.es == 2 && g.c_in <= 4 && lines <= 12 && line_elems <= 253 && g.w * g.c_in % 4 == 0 &&
         g.kt * g.kh * g.kw <= 64 && pool_ok;
}

// Bricks of 1 x 2 x 32 output voxels; halo rows of 4 channels (8 bytes).
Tiling small_tiling(const Geom &g) {
  Tiling t{};
  t.bt = 1;
  t.bh = 2;
  t.bw = 32;
  t.ht = g.kt;
  t.hh = g.sh + g.kh;
  t.hw = 31 * g.sw + g.kw;
  t.cc = 4;
  t.row = 8;
  t.slots = 64;
  t.nchunks = 1;
  return t;
}

// Voxel slots per workgroup of the item kernels: 128 (8 fragments of 16 per
// wave; two slots per lane in the exact fp32 kernel) or 64 (4 fragments; one
// slot per lane).  Wide bricks reuse each weight fragment
// over more voxels and stage less halo per output; narrow bricks double the
// workgroups, which pays when 128-slot bricks times 16-filter tiles give
// fewer waves than the GPU has SIMDs (the layer would otherwise need deep
// channel splits and their reduction pass), and for unpooled 16-bit layers
// well beyond that (their epilogue is then done in registers, without the
// LDS tile and its barriers).  Measured on MI355X over the
// C3D and R(2+1)D layers at batch 1 (and on the single fp32 layers).
// Tuning switch slots=64|128.
int brick_slots(const Geom &g) {
  {
    const int v = tune("slots");
    if (v == 64 || v == 128) return v;
  }
  const long voxels = static_cast<long>(std::max(g.n, 1)) * g.to * g.ho * g.wo;
  const long waves = (voxels + kSlots - 1) / kSlots * ((g.c_out + 15) / 16);
  // fp32 waves carry 8x the MFMA time per item (16x16x4 at 1/16 of the
  // 16-bit rate): narrow bricks only pay below one wave per CU.  16-bit
  // layers without pooling keep their narrow-tile epilogue in registers, so
  // narrow bricks pay there up to about eight 128-slot waves per SIMD.
  const bool pooled = g.qt * g.qh * g.qw > 1;
  const long limit = g.es == 4 ? 256 : (pooled ? 1024 : 8192);
  return waves < limit ? 64 : kSlots;
}

Tiling layer_tiling(const Geom &g) {
  return small_ok(g) ? small_tiling(g) : choose_tiling(g, brick_slots(g));
}

// mask of the 4x4 kernel block (p4, q4) at position pos (groups of 8 or 16
// are unions of 4x4 blocks that share their group's mask row).
struct Mask4 {
  const uint8_t *mask;
  int Q, ks, gm4, gn4;  // gm4 = g_m / 4
  // Optional order of the 4-filter blocks (g_m = 4 only): block p4 of the
  // layout is block perm[p4] of the layer.
  const int32_t *perm = nullptr;
  bool kept(int p4, int q4, int pos) const {
    const int p = perm ? perm[p4] : p4;
    return mask[(static_cast<size_t>(p / gm4) * Q + q4 / gn4) * ks + pos] == 1;
  }
};

// ---------------------------------------------------------------------------
// Kernel layouts
// ---------------------------------------------------------------------------

struct Layout {
  Plan plan{};
  uint32_t variant = 0;
  std::vector<uint32_t> step_ptr, item_ptr, items, keep;
  std::vector<uint8_t> a;  // operand stream, raw element bytes
};

// Element (filter m, channel c, position pos) of the dense weights, or zero
// when it lies outside the layer or is pruned.  Pruned weights are not read.
struct WeightSource {
  const uint8_t *w;
  const Geom &g;
  const Mask4 *m4;  // nullptr for dense
  void copy(uint8_t *dst, int m, int c, int pos) const {
    if (m < g.c_out && c < g.c_in && (!m4 || m4->kept(m / 4, c / 4, pos))) {
      const int mo = m4 && m4->perm ? 4 * m4->perm[m / 4] + (m & 3) : m;  // layer filter
      const size_t idx = (static_cast<size_t>(mo) * g.c_in + c) * g.ks + pos;
      std::memcpy(dst, w + idx * g.es, g.es);
    } else {
      std::memset(dst, 0, g.es);
    }
  }
};

struct Item {
  int ql, pos;
  uint32_t keep;
};

// Items of one chunk for one wave tile of 4*nb4 filters: every (block,
// position) that any of the tile's nb4 4x4 blocks keeps (all of them when
// dense), in position-major order.
std::vector<Item> chunk_items(const Geom &g, const Mask4 *m4, int cc, int ch, int p4_first,
                              int nb4 = 4) {
  std::vector<Item> out;
  const int blocks = cc / 4;
  const int q4_count = (g.c_in + 3) / 4;
  const int p4_count = (g.c_out + 3) / 4;
  for (int pos = 0; pos < g.ks; ++pos)
    for (int ql = 0; ql < blocks; ++ql) {
      const int q4 = ch * blocks + ql;
      if (q4 >= q4_count) continue;
      uint32_t keep = 0;
      for (int gi = 0; gi < nb4; ++gi) {
        const int p4 = p4_first + gi;
        if (p4 < p4_count && (!m4 || m4->kept(p4, q4, pos))) keep |= 1u << gi;
      }
      if (keep) out.push_back(Item{ql, pos, keep});
    }
  return out;
}

// LDS bank model of gfx950 (measured with a read-pattern probe): 64 banks of
// 4 bytes; a wave's ds_read_b64 is served in two passes of 32 lanes, and a
// pass takes as many cycles as its most loaded bank has distinct addresses.
// In the 16-bit item kernel a pass carries lane groups g and g+1, which read
// two different items for the same 16 voxel slots, so the planner pairs the
// items of each pass to avoid conflicts.
class PassCost {
 public:
  PassCost(const Geom &g, const Tiling &tl) : row_dw_(tl.row / 4) {
    for (int f = 0; f < tl.slots / 16; ++f)
      for (int n = 0; n < 16; ++n) {
        const int sl = 16 * f + n;
        const int tt = sl / (tl.bh * tl.bw), hh = (sl / tl.bw) % tl.bh, ww = sl % tl.bw;
        const int v = tt < tl.bt ? ((tt * g.st) * tl.hh + hh * g.sh) * tl.hw + ww * g.sw : 0;
        rows_.push_back(v);
      }
    span_ = tl.ht * tl.hh * tl.hw * row_dw_;
    memo_.assign(2 * static_cast<size_t>(span_) + 1, -1);
  }
  // Cycles of one pass whose two lane groups read byte offsets o1 and o2.
  int operator()(uint32_t o1, uint32_t o2) {
    const long d = (static_cast<long>(o2) - static_cast<long>(o1)) / 4;
    if (d < -span_ || d > span_) return eval(d);
    int8_t &m = memo_[static_cast<size_t>(d + span_)];
    if (m < 0) m = static_cast<int8_t>(eval(d));
    return m;
  }

 private:
  int eval(long d) const {
    int worst = 1;
    for (size_t f = 0; f < rows_.size(); f += 16) {
      long addr[64];
      int k = 0;
      for (int grp = 0; grp < 2; ++grp)
        for (int n = 0; n < 16; ++n)
          for (int e = 0; e < 2; ++e)
            addr[k++] = static_cast<long>(rows_[f + n]) * row_dw_ + (grp ? d : 0) + e;
      std::sort(addr, addr + 64);
      int per_bank[64] = {0};
      for (int i = 0; i < 64; ++i)
        if (i == 0 || addr[i] != addr[i - 1]) {
          const int b = static_cast<int>(((addr[i] % 64) + 64) % 64);
          worst = std::max(worst, ++per_bank[b]);
        }
    }
    return worst;
  }
  long row_dw_, span_;
  std::vector<int> rows_;
  std::vector<int8_t> memo_;
};

// Reorders a step-padded item list so that items 2k and 2k+1 share an LDS
// pass with as few bank conflicts as possible (greedy over a window), then
// lays the pairs out in K-step order: pass pairs (0,2) (4,6) (1,3) (5,7).
void pair_items(std::vector<Item> &its, const Geom &g, const Tiling &tl, PassCost &cost) {
  const size_t n = its.size();
  auto off = [&](const Item &it) { return it.ql < 0 ? 0u : item_offset(g, tl, it.ql, it.pos); };
  std::vector<char> used(n, 0);
  std::vector<Item> paired;
  paired.reserve(n);
  constexpr size_t kWindow = 48;
  for (size_t i = 0; i < n; ++i) {
    if (used[i]) continue;
    used[i] = 1;
    const uint32_t oi = off(its[i]);
    size_t best = n;
    int best_cost = 1 << 30;
    for (size_t j = i + 1, looked = 0; j < n && looked < kWindow; ++j) {
      if (used[j]) continue;
      ++looked;
      const int c = cost(oi, off(its[j]));
      if (c < best_cost) {
        best_cost = c;
        best = j;
        if (c == 1) break;
      }
    }
    paired.push_back(its[i]);
    if (best < n) {
      used[best] = 1;
      paired.push_back(its[best]);
    }
  }
  // n is a multiple of 8, so every item found a partner.
  for (size_t s = 0; s + 8 <= n; s += 8) {
    const Item *p = &paired[s];
    const Item step[8] = {p[0], p[2], p[1], p[3], p[4], p[6], p[5], p[7]};
    std::copy(step, step + 8, its.begin() + static_cast<long>(s));
  }
}

// KGS wave-tile width for the 16-bit item kernel: 1 (16 filters walk the
// union of their four 4x4 blocks' items), 2 (see below) or 4 (64 filters
// walk the union of sixteen blocks, each B fragment feeding four MFMAs, as
// in the dense kernel).  The wide union executes more zero-weight items but costs about
// 1/1.4 as much per item (measured over the C3D layers at batch 32: the
// narrow union runs at ~1.4x the dense kernel's time per executed item), so
// it wins when the narrow union already covers most items.  It is only
// considered where the dense kernel itself runs 64-filter tiles (256 filters
// or more) and either the layer gives every SIMD a 64-filter wave without
// channel splits, or its reduction is deep (K = c_in taps >= 8192) with at
// least 512 narrow waves (C3D conv4b-conv5b at batch 8-32, measured); at
// batch 1 the narrow tiles' extra waves matter more.
//
// Spatial-only 1x3x3 layers on 64-slot bricks with at least 1.25M outputs
// (voxels x filters) take 32-filter tiles instead (the union of eight
// blocks): measured at batch 1 on R(2+1)D layers 2-3 (-8% to -23%) and the
// S3D 64->192 layer (-7%), while 3x3x3, temporal and smaller layers ran
// slower with them.
int kgs_tile_width(const Geom &g, const Tiling &tl, const Mask4 *m4) {
  const long voxels = static_cast<long>(std::max(g.n, 1)) * g.to * g.ho * g.wo;
  if (g.es == 2 && m4 && tl.slots == 64 && g.kt == 1 && g.kh * g.kw == 9 &&
      voxels * g.c_out >= 1250000)
    return 2;
  if (g.es != 2 || !m4 || g.c_out < 256) return 1;
  const long bricks = (voxels + tl.slots - 1) / tl.slots;
  const bool deep = static_cast<long>(g.c_in) * g.kt * g.kh * g.kw >= 8192 &&
                    bricks * ((g.c_out + 15) / 16) >= 512;
  if (bricks * ((g.c_out + 63) / 64) < 1024 && !deep) return 1;
  double narrow = 0, wide = 0;
  const int p4_count = (g.c_out + 3) / 4;
  for (int ch = 0; ch < tl.nchunks; ++ch) {
    for (int p4 = 0; p4 < p4_count; p4 += 4)
      narrow += static_cast<double>(chunk_items(g, m4, tl.cc, ch, p4, 4).size());
    for (int p4 = 0; p4 < p4_count; p4 += 16)
      wide += 4.0 * static_cast<double>(chunk_items(g, m4, tl.cc, ch, p4, 16).size());
  }
  return wide < 1.4 * narrow ? 4 : 1;
}

// Channel splits trade per-workgroup fixed cost (prologue, first halo load,
// epilogue) and a reduction pass against parallelism.  The split count
// minimises a time model in cycles:
//   rounds * kFixed + chunks per workgroup * steps per chunk * step cycles
//   * (1 + kShare * (workgroups per CU - 1)) + [s > 1] (kReduce + partial
//   bytes written and read back / kPartialBytesPerCycle),
// with constants fitted to per-wave timestamps and per-layer traces of the
// C3D and R(2+1)D layers on MI355X.  wgs: workgroups of one split;
// per_cu_split / per_cu_whole: resident workgroups per CU of split and
// unsplit launches; cus: compute units.
int model_splits(const Geom &g, const Tiling &tl, int mfw, double chunk_steps, uint32_t variant,
                 long wgs, int per_cu_split, int per_cu_whole, long cus) {
  const long total_vox = static_cast<long>(g.n) * g.to * g.ho * g.wo;
  const double partial_bytes = 2.0 * static_cast<double>(total_vox) * ((g.c_out + 3) / 4 * 4) * 4;
  constexpr double kFixed = 12000, kReduce = 9600, kShare = 0.2, kPartialBytesPerCycle = 4200;
  // Pair steps read twice the items of a union step (an estimate until
  // measured per layer).
  const double step_cycles = variant == kVarKgsPair16 ? 600.0
                             : (mfw == 1 ? 380.0 : (mfw == 2 ? 555.0 : 815.0));
  // A chunk costs its K-steps, but no less than the exposed latency of its
  // halo load, plus the barriers and LDS commit around it.
  constexpr double kChunkLatency = 5000, kChunkFixed = 2000;
  const double chunk_cycles = std::max(chunk_steps * step_cycles, kChunkLatency) + kChunkFixed;
  int splits = 1;
  double best = -1;
  for (int s = 1; s <= tl.nchunks; ++s) {
    if (s > 1 && (tl.nchunks + s - 1) / s == (tl.nchunks + s - 2) / (s - 1)) continue;  // same chunks per WG
    const long n = wgs * s;
    const long per_cu = s > 1 ? per_cu_split : per_cu_whole;
    const long per = std::min<long>((n + cus - 1) / cus, per_cu);          // workgroups per CU at once
    const long rounds = (n + cus * per - 1) / (cus * per);
    const double t = rounds * (kFixed + ((tl.nchunks + s - 1) / s) * chunk_cycles *
                                            (1.0 + kShare * static_cast<double>(per - 1))) +
                     (s > 1 ? kReduce + s * partial_bytes / kPartialBytesPerCycle : 0.0);
    if (best < 0 || t < best) {
      best = t;
      splits = s;
    }
  }
  return splits;
}

// Filter rows (of 16) per wave tile of the item kernels, then the brick.
//
// Dense layers share every B fragment across the wave's rows, KGS layers walk
// the union of the tile's kernel groups' items (kgs_tile_width).  Dense: 64
// filters (4 rows) for layers of 256+ filters with >= 2000 output voxels,
// 16 (16-bit) for those with fewer than 256 (a few bricks, split many ways:
// at batch 1 C3D conv5a/b 14.7 -> 13.2 us, R(2+1)D layer 5 and S3D Mixed_5
// convs 5-10% faster), else 32; 16 for layers below 128 filters.  Layers of 128-255 filters take
// 32-filter tiles, dense or KGS, when that still leaves 2048 waves (two per
// SIMD): C3D conv2 at batch 1 dense 45.6 -> 38.7 us, KGS 40.9 -> 37.2 us, at
// batch 32 1022 -> 893 and 916 -> 847 us.  A wave tile of four rows runs
// on 64-slot bricks: on 128-slot bricks its accumulators and B ring exceed
// 256 registers and leave one wave per SIMD (16-bit; batch-32 conv3a/3b/4b
// 408/632/338 -> 350/597/309 us KGS, dense 410/643/340 -> 359/648/326 us).
// Two rows keep the brick width brick_slots chose: the kernel is held to
// two waves per SIMD there (a few spilled registers), and 128-slot bricks
// halve the weight loads per MFMA (C3D conv2 KGS batch 32 771 -> 693 us,
// dense 808 -> 723 us; batch 1 34.1 -> 33.0 us).
// Tuning switches dense_mfw, kgs_mfw and small_mfw override the width.
struct ItemPlan {
  Tiling tl;
  int mfw;
};

ItemPlan item_plan(const Geom &g, const Mask4 *m4, bool small) {
  ItemPlan ip{layer_tiling(g), 1};
  const bool dense = m4 == nullptr;
  if (small) {
    // Up to 32 filters per wave: wider tiles hold 4x the weights in
    // registers and drop residency to one wave per SIMD.
    ip.mfw = g.c_out > 16 ? 2 : 1;
    const int v = tune("small_mfw");
    if (v == 1 || v == 2) ip.mfw = v;
    return ip;
  }
  const long voxels = static_cast<long>(std::max(g.n, 1)) * g.to * g.ho * g.wo;
  const bool mid = g.es == 2 && g.c_out >= 128 && g.c_out < 256 &&
                   (voxels + 63) / 64 * ((g.c_out + 31) / 32) >= 2048;
  if (dense) {
    if (g.c_out >= 256) ip.mfw = voxels >= 2000 ? 4 : (g.es == 2 && voxels < 256 ? 1 : 2);
    else if (mid) ip.mfw = 2;
    // A shallow reduction (c_in taps < 4096) that the wide tiles would split
    // across workgroups runs unsplit on 16-filter tiles when those fill the
    // GPU without a split: the wide tiles' fp32 partials and reduction pass
    // cost more than the narrow tiles' unshared B fragments (batch 1: C3D
    // conv3a 32 -> 24 us, R(2+1)D layer-4 first spatial conv 17.6 -> 12.8 us,
    // S3D Mixed_4e/4f branch-1 spatial convs 13 -> 11 us; deeper layers such
    // as C3D conv3b ran slower unsplit).  Splits are judged by the launch
    // model at two resident workgroups per CU on 256 CUs.
    const long taps = static_cast<long>(g.c_in) * g.kt * g.kh * g.kw;
    if (g.es == 2 && g.c_out >= 256 && ip.mfw > 1 && taps < 4096) {
      auto splits_at = [&](int mfw) {
        const Tiling t = mfw >= 4 && ip.tl.slots == 128 ? choose_tiling(g, 64) : ip.tl;
        const long bricks = static_cast<long>(std::max(g.n, 1)) * ((g.to + t.bt - 1) / t.bt) *
                            ((g.ho + t.bh - 1) / t.bh) * ((g.wo + t.bw - 1) / t.bw);
        const long ntg = ((g.c_out + 16 * mfw - 1) / (16 * mfw) + 3) / 4;
        long steps = 0;
        for (int ch = 0; ch < t.nchunks; ++ch)
          steps += ((std::min(t.cc, g.c_in - ch * t.cc) + 3) / 4 * g.ks + 7) / 8;
        return model_splits(g, t, mfw, static_cast<double>(steps) / t.nchunks, kVarDenseItems16,
                            bricks * ntg, 2, 2, 256);
      };
      if (splits_at(ip.mfw) > 1 && splits_at(1) == 1) ip.mfw = 1;
    }
    const int v = tune("dense_mfw");
    if (v == 1 || v == 2 || v == 4) ip.mfw = v;
  } else {
    ip.mfw = mid ? 2 : kgs_tile_width(g, ip.tl, m4);
    const int v = tune("kgs_mfw");
    if (v == 1 || v == 2 || v == 4) ip.mfw = v;
  }
  if (g.es == 2 && ip.mfw >= 4 && ip.tl.slots == 128 && tune("slots") != 128)
    ip.tl = choose_tiling(g, 64);
  return ip;
}

// Order of the 4-filter blocks for a 16-bit union layout (g_m = 4): the
// blocks that share a wave tile should keep many of the same (channel block,
// position) items, since the tile multiplies the union of its blocks' items.
// Greedy (each tile grows by the block that adds the fewest new items to its
// union), then swaps of two blocks between two tiles that shrink the sum of
// the unions (a fixed pseudo-random sequence of candidate swaps, so packing
// is deterministic).  Returns layout block -> layer block, c_out / 4 entries.
std::vector<int32_t> cluster_blocks(const Geom &g, const Mask4 &m4, int tile_blocks) {
  const int P4 = g.c_out / 4, Q4 = (g.c_in + 3) / 4;
  const int words = (Q4 * g.ks + 63) / 64;
  std::vector<uint64_t> bits(static_cast<size_t>(P4) * words, 0);
  for (int p = 0; p < P4; ++p)
    for (int q = 0; q < Q4; ++q)
      for (int pos = 0; pos < g.ks; ++pos)
        if (m4.kept(p, q, pos)) {
          const int b = q * g.ks + pos;
          bits[static_cast<size_t>(p) * words + b / 64] |= 1ull << (b % 64);
        }
  auto row = [&](int p) { return &bits[static_cast<size_t>(p) * words]; };
  auto union_size = [&](const int32_t *members, int n) {
    int total = 0;
    for (int w = 0; w < words; ++w) {
      uint64_t u = 0;
      for (int k = 0; k < n; ++k) u |= row(members[k])[w];
      total += __builtin_popcountll(u);
    }
    return total;
  };
  std::vector<int32_t> order;
  order.reserve(P4);
  std::vector<char> used(P4, 0);
  std::vector<uint64_t> acc(words);
  for (int t0 = 0; t0 < P4; t0 += tile_blocks) {
    int seed = 0;
    while (used[seed]) ++seed;
    used[seed] = 1;
    order.push_back(seed);
    std::copy(row(seed), row(seed) + words, acc.begin());
    for (int k = 1; k < tile_blocks && t0 + k < P4; ++k) {
      int best = -1, best_add = 0;
      for (int p = 0; p < P4; ++p) {
        if (used[p]) continue;
        int add = 0;
        for (int w = 0; w < words; ++w) add += __builtin_popcountll(row(p)[w] & ~acc[w]);
        if (best < 0 || add < best_add) best = p, best_add = add;
      }
      used[best] = 1;
      order.push_back(best);
      for (int w = 0; w < words; ++w) acc[w] |= row(best)[w];
    }
  }
  const int tiles = (P4 + tile_blocks - 1) / tile_blocks;
  if (tiles > 1) {
    uint64_t lcg = 0x9E3779B97F4A7C15ull;
    auto next = [&](int n) {
      lcg = lcg * 6364136223846793005ull + 1442695040888963407ull;
      return static_cast<int>((lcg >> 33) % static_cast<uint64_t>(n));
    };
    auto tile_n = [&](int t) { return std::min(tile_blocks, P4 - t * tile_blocks); };
    std::vector<int32_t> ta(tile_blocks), tb(tile_blocks);
    for (int it = 0; it < 40 * P4; ++it) {
      const int a = next(tiles), b = next(tiles);
      if (a == b) continue;
      const int na = tile_n(a), nb = tile_n(b);
      const int i = next(na), j = next(nb);
      int32_t *pa = &order[static_cast<size_t>(a) * tile_blocks];
      int32_t *pb = &order[static_cast<size_t>(b) * tile_blocks];
      std::copy(pa, pa + na, ta.begin());
      std::copy(pb, pb + nb, tb.begin());
      std::swap(ta[i], tb[j]);
      if (union_size(ta.data(), na) + union_size(tb.data(), nb) <
          union_size(pa, na) + union_size(pb, nb))
        std::swap(pa[i], pb[j]);
    }
  }
  return order;
}

// K-steps of a union layout: every wave tile's items of every chunk, padded
// to whole steps.
long union_steps(const Geom &g, const Tiling &tl, const Mask4 &m4, int mfw) {
  const int wt_count = (g.c_out + 16 * mfw - 1) / (16 * mfw);
  long steps = 0;
  for (int wt = 0; wt < wt_count; ++wt)
    for (int ch = 0; ch < tl.nchunks; ++ch)
      steps += (static_cast<long>(chunk_items(g, &m4, tl.cc, ch, wt * 4 * mfw, 4 * mfw).size()) + 7) / 8;
  return steps;
}

// 16-bit MFMA item layout (variants kVarDenseItems16, kVarKgsUnion16) and
// the f32 16x16x4 dense layout (kVarDenseItemsF32).  For kVarKgsUnion16 the
// 4-filter blocks may be reordered (cluster_blocks) when that saves enough
// K-steps; the keep section then maps each wave tile's block slots to layer
// blocks.

void build_items_layout(const Geom &g, const Tiling &tl, const uint8_t *w, const Mask4 *m4,
                        Layout &L, bool small, int mfw) {
  const bool f32 = g.es == 4;
  const int ips = f32 ? 4 : 8;           // items per K-step
  const int epl = f32 ? 4 : 8;           // operand elements per lane
  const bool dense = m4 == nullptr;
  const int wt_count = (g.c_out + 16 * mfw - 1) / (16 * mfw);
  L.variant = small ? (dense ? kVarSmallDense16 : kVarSmallKgs16)
                    : (dense ? (f32 ? kVarDenseItemsF32 : kVarDenseItems16)
                             : (f32 ? kVarKgsUnionF32 : kVarKgsUnion16));
  L.plan.mfw = mfw;
  L.plan.wave_tiles = wt_count;
  L.plan.items_per_step = ips;
  L.step_ptr.assign(static_cast<size_t>(wt_count) * (tl.nchunks + 1), 0);
  L.item_ptr.assign(wt_count, 0);
  Mask4 reordered{};
  std::vector<int32_t> perm;
  // Used when it saves at least 5% of the K-steps (tuning switch
  // kgs_order=1: any saving, 0: never): a reordered tile's four lane groups
  // store four separate 8-byte pieces per voxel instead of 32 contiguous
  // bytes, which ate the 3% that i.i.d. KGS masks gain (whole-group vanilla
  // masks cluster better: 11%, 1.5-2.3% faster).
  const int order = tune("kgs_order");
  if (!dense && !f32 && !small && m4->gm4 == 1 && g.c_out % 4 == 0 && wt_count > 1 &&
      order != 0) {
    perm = cluster_blocks(g, *m4, 4 * mfw);
    reordered = *m4;
    reordered.perm = perm.data();
    const long natural = union_steps(g, tl, *m4, mfw);
    const long clustered = union_steps(g, tl, reordered, mfw);
    if (order == 1 ? clustered < natural : clustered <= natural - natural / 20) {
      m4 = &reordered;
      L.plan.gmap = 1;
      const int P4 = g.c_out / 4;
      for (int b = 0; b < wt_count * 4 * mfw; ++b)
        L.keep.push_back(static_cast<uint32_t>(b < P4 ? perm[b] : b));
    }
  }
  WeightSource src{w, g, m4};

  PassCost cost(g, tl);
  auto prepare = [&](std::vector<Item> its) {
    while (its.size() % ips) its.push_back(Item{-1, 0, 0});  // zero-weight filler
    if (!f32) pair_items(its, g, tl, cost);
    return its;
  };
  // Dense: one item list shared by every wave tile.
  std::vector<std::vector<Item>> shared;
  if (dense)
    for (int ch = 0; ch < tl.nchunks; ++ch)
      shared.push_back(prepare(chunk_items(g, nullptr, tl.cc, ch, 0)));

  uint32_t step = 0;
  for (int wt = 0; wt < wt_count; ++wt) {
    const uint32_t first_step = step;
    const bool write_items = !dense || wt == 0;
    L.item_ptr[wt] = dense ? 0 : first_step;
    for (int ch = 0; ch < tl.nchunks; ++ch) {
      L.step_ptr[static_cast<size_t>(wt) * (tl.nchunks + 1) + ch] = step;
      const std::vector<Item> its =
          dense ? shared[ch] : prepare(chunk_items(g, m4, tl.cc, ch, wt * 4 * mfw, 4 * mfw));
      const int nsteps = static_cast<int>(its.size()) / ips;
      for (int s = 0; s < nsteps; ++s) {
        const Item *si = &its[static_cast<size_t>(s) * ips];
        if (write_items)
          for (int e = 0; e < ips; ++e)
            L.items.push_back(si[e].ql < 0 ? 0u : item_offset(g, tl, si[e].ql, si[e].pos));
        // A operand for this step, MFMA lane order.
        const size_t base = L.a.size();
        L.a.resize(base + static_cast<size_t>(mfw) * 64 * epl * g.es);
        uint8_t *dst = L.a.data() + base;
        for (int i = 0; i < mfw; ++i)
          for (int lane = 0; lane < 64; ++lane)
            for (int e = 0; e < epl; ++e) {
              const int m = wt * 16 * mfw + 16 * i + (lane & 15);
              const int lg = lane >> 4;
              // 16-bit: lane group lg holds items 2lg, 2lg+1, 4 channels each.
              // f32: lane group lg holds item lg, element e = channel e.
              const Item &it = f32 ? si[lg] : si[2 * lg + e / 4];
              const int cin = f32 ? e : e % 4;
              uint8_t *out = dst + ((static_cast<size_t>(i) * 64 + lane) * epl + e) * g.es;
              if (it.ql < 0) {
                std::memset(out, 0, g.es);
              } else {
                const int c = 4 * (ch * (tl.cc / 4) + it.ql) + cin;
                src.copy(out, m, c, it.pos);
              }
            }
        ++step;
      }
    }
    L.step_ptr[static_cast<size_t>(wt) * (tl.nchunks + 1) + tl.nchunks] = step;
    L.plan.tile_steps = std::max<int32_t>(L.plan.tile_steps, static_cast<int32_t>(step - first_step));
  }
}

// ---------------------------------------------------------------------------
// Pair mapping (kVarKgsPair16): two items per 2:4 sparse MFMA slot
// ---------------------------------------------------------------------------

struct ItemPair {
  Item x, y;  // y.ql < 0: no partner (an offset-0 read that no group keeps)
};

// Pairs the items of one 16-filter tile and chunk so that no kernel group of
// the tile keeps both items of a pair: a filter row then has at most two
// nonzero weights in every quad (X.c0, X.c1, Y.c0, Y.c1) and (X.c2, X.c3,
// Y.c2, Y.c3), the 2:4 pattern the sparse MFMA multiplies at twice the dense
// rate.  Greedy, most constrained items first: an item kept by all four
// groups has no partner; one kept by three groups can only take an item kept
// by the fourth group alone; one kept by two groups takes the complementary
// two groups first, then an item of either other group alone; items kept by
// one group pair across groups, largest buckets first.  Every item lands in
// exactly one pair.
std::vector<ItemPair> pair_up_wide(const std::vector<Item> &items);

std::vector<ItemPair> pair_up(const std::vector<Item> &items, int groups = 4) {
  if (groups > 4) return pair_up_wide(items);
  std::vector<Item> b[16];
  for (const Item &it : items) b[it.keep & 15u].push_back(it);
  std::vector<ItemPair> out;
  out.reserve(items.size());
  const Item none{-1, 0, 0};
  auto take = [&](int m) {
    const Item it = b[m].back();
    b[m].pop_back();
    return it;
  };
  while (!b[15].empty()) out.push_back({take(15), none});
  for (const int m : {7, 11, 13, 14}) {
    const int c = 15 & ~m;
    while (!b[m].empty() && !b[c].empty()) out.push_back({take(m), take(c)});
    while (!b[m].empty()) out.push_back({take(m), none});
  }
  for (const int m : {3, 5, 6})
    while (!b[m].empty() && !b[15 & ~m].empty()) out.push_back({take(m), take(15 & ~m)});
  for (const int m : {3, 5, 6, 9, 10, 12}) {
    const int c = 15 & ~m, s1 = c & -c, s2 = c & ~s1;
    while (!b[m].empty()) {
      const int pick = b[s1].size() >= b[s2].size() ? s1 : s2;
      if (b[pick].empty()) out.push_back({take(m), none});
      else out.push_back({take(m), take(pick)});
    }
  }
  for (;;) {
    int s[4] = {1, 2, 4, 8};
    std::sort(s, s + 4, [&](int u, int v) { return b[u].size() > b[v].size(); });
    if (b[s[1]].empty()) break;
    out.push_back({take(s[0]), take(s[1])});
  }
  for (const int m : {1, 2, 4, 8})
    while (!b[m].empty()) out.push_back({take(m), none});
  // Ascending by position, then channel block: neighbouring pairs read
  // nearby halo rows.
  std::stable_sort(out.begin(), out.end(), [](const ItemPair &u, const ItemPair &v) {
    return u.x.pos != v.x.pos ? u.x.pos < v.x.pos : u.x.ql < v.x.ql;
  });
  return out;
}

// Pairing for wide tiles (8 or 16 kernel groups): most constrained first --
// items in decreasing order of how many groups keep them, each taking the
// disjoint partner kept by the most groups (greedy matching).
std::vector<ItemPair> pair_up_wide(const std::vector<Item> &items) {
  const size_t n = items.size();
  std::vector<size_t> order(n);
  std::iota(order.begin(), order.end(), 0);
  auto pc = [&](size_t i) { return __builtin_popcount(items[i].keep); };
  std::stable_sort(order.begin(), order.end(), [&](size_t u, size_t v) { return pc(u) > pc(v); });
  std::vector<char> used(n, 0);
  std::vector<ItemPair> out;
  out.reserve(n);
  const Item none{-1, 0, 0};
  for (size_t a = 0; a < n; ++a) {
    const size_t i = order[a];
    if (used[i]) continue;
    used[i] = 1;
    size_t best = n;
    int best_pc = -1;
    for (size_t b = a + 1; b < n; ++b) {
      const size_t j = order[b];
      if (used[j] || (items[i].keep & items[j].keep)) continue;
      if (pc(j) > best_pc) {
        best_pc = pc(j);
        best = j;
      }
    }
    if (best < n) {
      used[best] = 1;
      out.push_back({items[i], items[best]});
    } else {
      out.push_back({items[i], none});
    }
  }
  std::stable_sort(out.begin(), out.end(), [](const ItemPair &u, const ItemPair &v) {
    return u.x.pos != v.x.pos ? u.x.pos < v.x.pos : u.x.ql < v.x.ql;
  });
  return out;
}

// Lays out a padded pair list (a multiple of 8 pairs) step by step.  In a
// step, lane groups g and g + 1 (g even) read pairs (g, g + 1) and (g + 4,
// g + 5) in the same LDS passes, so the list is regrouped into couples of
// pairs whose items are read together with few bank conflicts (greedy over a
// window; a couple may swap the roles X and Y of its second pair).
void couple_pairs(std::vector<ItemPair> &prs, const Geom &g, const Tiling &tl, PassCost &cost) {
  const size_t n = prs.size();
  auto off = [&](const Item &it) { return it.ql < 0 ? 0u : item_offset(g, tl, it.ql, it.pos); };
  std::vector<char> used(n, 0);
  std::vector<ItemPair> out;
  out.reserve(n);
  constexpr size_t kWindow = 32;
  for (size_t i = 0; i < n; ++i) {
    if (used[i]) continue;
    used[i] = 1;
    const uint32_t px = off(prs[i].x), py = off(prs[i].y);
    size_t best = n;
    bool best_swap = false;
    int best_cost = 1 << 30;
    for (size_t j = i + 1, looked = 0; j < n && looked < kWindow; ++j) {
      if (used[j]) continue;
      ++looked;
      const uint32_t qx = off(prs[j].x), qy = off(prs[j].y);
      const int straight = cost(px, qx) + cost(py, qy);
      const int swapped = cost(px, qy) + cost(py, qx);
      const int c = std::min(straight, swapped);
      if (c < best_cost) {
        best_cost = c;
        best = j;
        best_swap = swapped < straight;
        if (c == 2) break;
      }
    }
    out.push_back(prs[i]);
    if (best < n) {
      used[best] = 1;
      ItemPair q = prs[best];
      if (best_swap) std::swap(q.x, q.y);
      out.push_back(q);
    }
  }
  // Consecutive couples fill each step's positions (0,1) (2,3) (4,5) (6,7):
  // lane groups 0/1 and 2/3 share a pass, pairs 0-3 are read by reads 0-1
  // and pairs 4-7 by reads 2-3.
  prs.swap(out);
}

// Pair layout: per 16-filter tile and chunk the paired items, 8 pairs per
// K-step; per step 16 LDS offsets (lane group g: X and Y of pairs g and
// g + 4), the step's kept 4x4 weight blocks, 32 bytes each ([row][channel])
// in (pair, group) order, and per (lane group g, kernel group) a descriptor
// {byte offset of the block of pair 2g, of pair 2g + 1 (2^31 when the group
// keeps neither item), index register, 0}.  The index register holds two
// bits per compressed A element: (0, 1, 0, 1) = 0x44 selects X's channels of
// a pair's two quads, (2, 3, 2, 3) = 0xEE selects Y's; pair 2g sits in bits
// 0-7, pair 2g + 1 in bits 8-15.
//
// Wide tiles (mfw = 2 or 4: 32 or 64 filters, 8 or 16 kernel groups sharing
// every B fragment): the pairs are disjoint over all the tile's groups, and
// the weights stream in MFMA lane order, [step][16-filter row i][lane][8]
// (zeros where a group keeps neither item of a pair), with the index
// registers [step][i][lane] in the descriptor section.
void build_pairs_layout(const Geom &g, const Tiling &tl, const uint8_t *w, const Mask4 *m4,
                        Layout &L, int mfw) {
  const int wt_count = (g.c_out + 16 * mfw - 1) / (16 * mfw);
  L.variant = kVarKgsPair16;
  L.plan.mfw = mfw;
  L.plan.wave_tiles = wt_count;
  L.plan.items_per_step = 16;
  L.step_ptr.assign(static_cast<size_t>(wt_count) * (tl.nchunks + 1), 0);
  L.item_ptr.assign(wt_count, 0);
  WeightSource src{w, g, m4};
  PassCost cost(g, tl);
  auto off = [&](const Item &it) { return it.ql < 0 ? 0u : item_offset(g, tl, it.ql, it.pos); };
  const Item none{-1, 0, 0};
  uint32_t step = 0, blocks = 0;
  for (int wt = 0; wt < wt_count; ++wt) {
    const uint32_t first = step;
    L.item_ptr[wt] = first;
    for (int ch = 0; ch < tl.nchunks; ++ch) {
      L.step_ptr[static_cast<size_t>(wt) * (tl.nchunks + 1) + ch] = step;
      std::vector<ItemPair> prs =
          pair_up(chunk_items(g, m4, tl.cc, ch, wt * 4 * mfw, 4 * mfw), 4 * mfw);
      while (prs.size() % 8) prs.push_back({none, none});
      couple_pairs(prs, g, tl, cost);
      for (size_t s0 = 0; s0 < prs.size(); s0 += 8, ++step) {
        const ItemPair *sp = &prs[s0];
        for (int lg = 0; lg < 4; ++lg) {
          L.items.push_back(off(sp[lg].x));
          L.items.push_back(off(sp[lg].y));
          L.items.push_back(off(sp[lg + 4].x));
          L.items.push_back(off(sp[lg + 4].y));
        }
        if (mfw > 1) {
          // lane (m, ga) of row i: pairs 2ga, 2ga + 1 -> A elements 0-3, 4-7
          const size_t base = L.a.size();
          L.a.resize(base + static_cast<size_t>(mfw) * 64 * 8 * g.es);
          for (int i = 0; i < mfw; ++i)
            for (int lane = 0; lane < 64; ++lane) {
              const int blk = 4 * i + ((lane & 15) >> 2);       // 4x4 block in the tile
              const int m = wt * 16 * mfw + 16 * i + (lane & 15);
              uint32_t idx = 0;
              for (int h = 0; h < 2; ++h) {
                const ItemPair &pr = sp[2 * (lane >> 4) + h];
                const bool ky = (pr.y.keep >> blk) & 1u;
                const bool kx = (pr.x.keep >> blk) & 1u;
                idx |= (ky ? 0xEEu : 0x44u) << (8 * h);
                uint8_t *dst = L.a.data() + base + ((static_cast<size_t>(i) * 64 + lane) * 8 + 4 * h) * g.es;
                for (int c = 0; c < 4; ++c) {
                  if (kx || ky) {
                    const Item &it = ky ? pr.y : pr.x;
                    src.copy(dst + c * g.es, m, 4 * (ch * (tl.cc / 4) + it.ql) + c, it.pos);
                  } else {
                    std::memset(dst + c * g.es, 0, g.es);
                  }
                }
              }
              L.keep.push_back(idx);
            }
          continue;
        }
        uint32_t keep = 0, side = 0;
        for (int j = 0; j < 8; ++j)
          for (int gi = 0; gi < 4; ++gi) {
            const bool kx = (sp[j].x.keep >> gi) & 1u, ky = (sp[j].y.keep >> gi) & 1u;
            if (kx || ky) keep |= 1u << (4 * j + gi);
            if (ky) side |= 1u << (4 * j + gi);
          }
        for (int lg = 0; lg < 4; ++lg)
          for (int gi = 0; gi < 4; ++gi) {
            uint32_t off[2], idx = 0;
            for (int h = 0; h < 2; ++h) {
              const int b = 4 * (2 * lg + h) + gi;
              const uint32_t below = static_cast<uint32_t>(__builtin_popcount(keep & ((1u << b) - 1u)));
              off[h] = ((keep >> b) & 1u) ? (blocks + below) * 32u : 0x80000000u;
              idx |= (((side >> b) & 1u) ? 0xEEu : 0x44u) << (8 * h);
            }
            L.keep.push_back(off[0]);
            L.keep.push_back(off[1]);
            L.keep.push_back(idx);
            L.keep.push_back(0);
          }
        for (int b = 0; b < 32; ++b) {
          if (!((keep >> b) & 1u)) continue;
          const int j = b >> 2, gi = b & 3;
          const Item &it = ((side >> b) & 1u) ? sp[j].y : sp[j].x;
          const size_t base = L.a.size();
          L.a.resize(base + 16 * static_cast<size_t>(g.es));
          for (int r = 0; r < 4; ++r)
            for (int c = 0; c < 4; ++c)
              src.copy(L.a.data() + base + (r * 4 + c) * g.es, wt * 16 + 4 * gi + r,
                       4 * (ch * (tl.cc / 4) + it.ql) + c, it.pos);
          ++blocks;
        }
      }
    }
    L.step_ptr[static_cast<size_t>(wt) * (tl.nchunks + 1) + tl.nchunks] = step;
    L.plan.tile_steps = std::max<int32_t>(L.plan.tile_steps, static_cast<int32_t>(step - first));
  }
  // check_desc bounds a layer to 1e9 weights, so the kept blocks (16 weights
  // each) end below byte 2^31: every kept offset stays below the not-kept mark.
}

// Block-pair layout (kVarKgsBlockPair16): the two items of a 2:4 slot are the
// channel blocks 2i and 2i + 1 at one kernel position, which the kernel
// stages interleaved so that one 16-byte LDS read is the slot's operand.  A
// kernel group takes block 2i if it keeps it, else block 2i + 1 if it keeps
// that; groups keeping both get block 2i + 1 in a second slot.  Per step 8
// slots: 8 LDS offsets (lane group g: slots g and g + 4), the weights in MFMA
// lane order [step][lane][8] and the index registers [step][lane].
void build_block_pairs_layout(const Geom &g, const Tiling &tl, const uint8_t *w, const Mask4 *m4,
                              Layout &L) {
  const int wt_count = (g.c_out + 15) / 16;
  L.variant = kVarKgsBlockPair16;
  L.plan.mfw = 1;
  L.plan.wave_tiles = wt_count;
  L.plan.items_per_step = 16;
  L.step_ptr.assign(static_cast<size_t>(wt_count) * (tl.nchunks + 1), 0);
  L.item_ptr.assign(wt_count, 0);
  WeightSource src{w, g, m4};
  const int q4_count = (g.c_in + 3) / 4, p4_count = (g.c_out + 3) / 4;
  struct Slot {
    uint32_t off;
    int q4x, pos;
    uint8_t sel[4];  // per kernel group: 0 none, 1 block 2i, 2 block 2i + 1
  };
  uint32_t step = 0;
  for (int wt = 0; wt < wt_count; ++wt) {
    const uint32_t first = step;
    L.item_ptr[wt] = first;
    for (int ch = 0; ch < tl.nchunks; ++ch) {
      L.step_ptr[static_cast<size_t>(wt) * (tl.nchunks + 1) + ch] = step;
      std::vector<Slot> slots;
      for (int pos = 0; pos < g.ks; ++pos)
        for (int i = 0; i < tl.cc / 8; ++i) {
          const int qx = ch * (tl.cc / 4) + 2 * i, qy = qx + 1;
          uint32_t kx = 0, ky = 0;
          for (int gi = 0; gi < 4; ++gi) {
            const int p4 = wt * 4 + gi;
            if (p4 >= p4_count) continue;
            if (qx < q4_count && m4->kept(p4, qx, pos)) kx |= 1u << gi;
            if (qy < q4_count && m4->kept(p4, qy, pos)) ky |= 1u << gi;
          }
          if (!(kx | ky)) continue;
          Slot s1{item_offset(g, tl, 2 * i, pos), qx, pos, {0, 0, 0, 0}};
          Slot s2 = s1;
          for (int gi = 0; gi < 4; ++gi) {
            s1.sel[gi] = ((kx >> gi) & 1u) ? 1 : (((ky >> gi) & 1u) ? 2 : 0);
            s2.sel[gi] = ((kx & ky) >> gi) & 1u ? 2 : 0;
          }
          slots.push_back(s1);
          if (kx & ky) slots.push_back(s2);
        }
      while (slots.size() % 8) slots.push_back(Slot{0, -1, 0, {0, 0, 0, 0}});
      for (size_t s0 = 0; s0 < slots.size(); s0 += 8, ++step) {
        const Slot *sp = &slots[s0];
        for (int lg = 0; lg < 4; ++lg) {
          L.items.push_back(sp[lg].off);
          L.items.push_back(sp[lg + 4].off);
        }
        const size_t base = L.a.size();
        L.a.resize(base + 64 * 8 * static_cast<size_t>(g.es));
        for (int lane = 0; lane < 64; ++lane) {
          const int gi = (lane & 15) >> 2, m = wt * 16 + (lane & 15);
          uint32_t idx = 0;
          for (int h = 0; h < 2; ++h) {
            const Slot &sl = sp[2 * (lane >> 4) + h];
            const int sel = sl.q4x < 0 ? 0 : sl.sel[gi];
            idx |= (sel == 2 ? 0xEEu : 0x44u) << (8 * h);
            uint8_t *dst = L.a.data() + base + (static_cast<size_t>(lane) * 8 + 4 * h) * g.es;
            for (int c = 0; c < 4; ++c) {
              if (sel == 0) std::memset(dst + c * g.es, 0, g.es);
              else src.copy(dst + c * g.es, m, 4 * (sl.q4x + sel - 1) + c, sl.pos);
            }
          }
          L.keep.push_back(idx);
        }
      }
    }
    L.step_ptr[static_cast<size_t>(wt) * (tl.nchunks + 1) + tl.nchunks] = step;
    L.plan.tile_steps = std::max<int32_t>(L.plan.tile_steps, static_cast<int32_t>(step - first));
  }
}

// Exact f32 KGS layout (kVarKgsExactF32): per 16-filter tile and chunk, the
// union items with their kept-group bits and one 64-float A column set each
// (lane l = 4*(4*group + channel) + row).
void build_exact_f32_layout(const Geom &g, const Tiling &tl, const uint8_t *w, const Mask4 *m4,
                            Layout &L) {
  const int wt_count = (g.c_out + 15) / 16;
  L.variant = kVarKgsExactF32;
  L.plan.mfw = 1;
  L.plan.wave_tiles = wt_count;
  L.plan.items_per_step = 1;
  L.step_ptr.assign(static_cast<size_t>(wt_count) * (tl.nchunks + 1), 0);
  L.item_ptr.assign(wt_count, 0);
  WeightSource src{w, g, m4};
  uint32_t item = 0;
  for (int wt = 0; wt < wt_count; ++wt) {
    L.item_ptr[wt] = item;
    for (int ch = 0; ch < tl.nchunks; ++ch) {
      L.step_ptr[static_cast<size_t>(wt) * (tl.nchunks + 1) + ch] = item;
      for (const Item &it : chunk_items(g, m4, tl.cc, ch, wt * 4)) {
        L.items.push_back(item_offset(g, tl, it.ql, it.pos));
        L.keep.push_back(it.keep);
        const size_t base = L.a.size();
        L.a.resize(base + 64 * 4);
        for (int lane = 0; lane < 64; ++lane) {
          const int blk = lane >> 2, row = lane & 3;
          const int gi = blk >> 2, cin = blk & 3;
          const int m = wt * 16 + 4 * gi + row;
          const int c = 4 * (ch * (tl.cc / 4) + it.ql) + cin;
          uint8_t *out = L.a.data() + base + lane * 4;
          if (it.keep & (1u << gi)) src.copy(out, m, c, it.pos);
          else std::memset(out, 0, 4);
        }
        ++item;
      }
    }
    L.step_ptr[static_cast<size_t>(wt) * (tl.nchunks + 1) + tl.nchunks] = item;
    L.plan.tile_steps = std::max<int32_t>(L.plan.tile_steps,
                                          static_cast<int32_t>(item - L.item_ptr[wt]));
  }
}

// Assemble header + canonical + layout sections.  With out == nullptr only
// the size is computed.
struct Sections {
  uint64_t header, canon[4], step_ptr, item_ptr, items, keep, a, total;
};

Sections section_offsets(const Canon *c, int es, const Layout &L) {
  Sections s{};
  uint64_t off = align_up(sizeof(rt3d_pack_info), kAlign);
  s.header = 0;
  if (c) {
    const uint64_t sz[4] = {c->group_ptr.size() * 4, c->pos.size() * 2, c->val_ptr.size() * 8,
                            c->nvals * static_cast<uint64_t>(es)};
    for (int i = 0; i < 4; ++i) {
      s.canon[i] = off;
      off = align_up(off + sz[i], kAlign);
    }
  }
  s.step_ptr = off;
  off = align_up(off + L.step_ptr.size() * 4, kAlign);
  s.item_ptr = off;
  off = align_up(off + L.item_ptr.size() * 4, kAlign);
  s.items = off;
  off = align_up(off + L.items.size() * 4, kAlign);
  s.keep = off;
  off = align_up(off + L.keep.size() * 4, kAlign);
  s.a = off;
  off = align_up(off + L.a.size(), kAlign);
  s.total = off;
  return s;
}

void fill_info(const rt3d_conv3d_desc *d, const Canon *c, const Layout &L, const Tiling &tl,
               const Sections &s, bool vanilla, rt3d_pack_info *info) {
  std::memset(info, 0, sizeof(*info));
  info->magic = kMagic;
  info->version = kVersion;
  info->desc_hash = desc_hash(d);
  info->variant = L.variant;
  info->tile_groups = 4;
  info->vanilla = vanilla ? 1 : 0;
  info->packed_bytes = s.total;
  if (c) {
    const uint64_t sz[4] = {c->group_ptr.size() * 4, c->pos.size() * 2, c->val_ptr.size() * 8,
                            c->nvals * static_cast<uint64_t>(esize_of(d->dtype))};
    for (int i = 0; i < 4; ++i) {
      info->canon_off[i] = s.canon[i];
      info->canon_bytes[i] = sz[i];
    }
    info->kept_positions = c->pos.size();
    info->kept_weights = c->nvals;
  } else {
    info->kept_positions = 0;
    info->kept_weights = static_cast<uint64_t>(d->c_out) * d->c_in * d->kt * d->kh * d->kw;
  }
  info->derived_off = s.step_ptr;
  info->derived_bytes = s.total - s.step_ptr;
  Plan p = L.plan;
  p.tiling = tl;
  p.step_ptr_off = s.step_ptr;
  p.item_ptr_off = s.item_ptr;
  p.items_off = s.items;
  p.a_off = s.a;
  p.keep_off = s.keep;
  std::memcpy(info->plan, &p, sizeof(p));
}

void write_blob(uint8_t *out, const rt3d_pack_info &info, const Canon *c, const uint8_t *w,
                const rt3d_conv3d_desc *d, const Layout &L, const Sections &s) {
  std::memset(out, 0, s.total);
  std::memcpy(out, &info, sizeof(info));
  if (c) {
    std::memcpy(out + s.canon[0], c->group_ptr.data(), c->group_ptr.size() * 4);
    std::memcpy(out + s.canon[1], c->pos.data(), c->pos.size() * 2);
    std::memcpy(out + s.canon[2], c->val_ptr.data(), c->val_ptr.size() * 8);
    // vals: group (p, q), rows i (filter), then j (channel), then kept r.
    const int es = esize_of(d->dtype);
    const int ks = d->kt * d->kh * d->kw;
    uint8_t *vals = out + s.canon[3];
    for (int p = 0; p < c->P; ++p) {
      const int gm = std::min(d->g_m, d->c_out - p * d->g_m);
      for (int q = 0; q < c->Q; ++q) {
        const int gn = std::min(d->g_n, d->c_in - q * d->g_n);
        const size_t gi = static_cast<size_t>(p) * c->Q + q;
        const uint32_t k0 = c->group_ptr[gi], k = c->group_ptr[gi + 1] - k0;
        uint8_t *dst = vals + c->val_ptr[gi] * es;
        for (int i = 0; i < gm; ++i)
          for (int j = 0; j < gn; ++j)
            for (uint32_t r = 0; r < k; ++r) {
              const size_t widx =
                  (static_cast<size_t>(p * d->g_m + i) * d->c_in + q * d->g_n + j) * ks + c->pos[k0 + r];
              std::memcpy(dst + ((static_cast<size_t>(i) * gn + j) * k + r) * es, w + widx * es, es);
            }
      }
    }
  }
  std::memcpy(out + s.step_ptr, L.step_ptr.data(), L.step_ptr.size() * 4);
  std::memcpy(out + s.item_ptr, L.item_ptr.data(), L.item_ptr.size() * 4);
  if (!L.items.empty()) std::memcpy(out + s.items, L.items.data(), L.items.size() * 4);
  if (!L.keep.empty()) std::memcpy(out + s.keep, L.keep.data(), L.keep.size() * 4);
  if (!L.a.empty()) std::memcpy(out + s.a, L.a.data(), L.a.size());
}

// 16-bit KGS mapping: pairs (2:4 sparse MFMA over 64-slot bricks) or the
// union of a tile's kept items.  Tuning switch kgs_map=0 (union) or 1
// (pairs).  The union is the default: on MI355X a K-step's cost follows its
// LDS read instructions and address arithmetic, and a pair step reads every
// item of the union as well (two 8-byte reads per pair per voxel fragment)
// plus the register moves that interleave them, so halving the MFMAs does
// not pay (measured on every C3D layer at batch 1 and 32).
bool use_pairs(const Geom &g, const Mask4 *m4) {
  (void)m4;
  if (g.es != 2) return false;
  return tune("kgs_map") == 1;
}

// fp32 KGS: the exact 4x4x1 kernel (only kept blocks are multiplied; one
// loop iteration per item), or the dense 16x16x4 kernel over the union of
// each 16-filter tile's kept items (pruned entries multiplied as zeros; one
// iteration per four items).  The exact kernel wins whenever its MFMA work
// matters (config 2, 256->256: 162 against 220 us; every C3D layer); a layer
// whose kept MACs take under 5 us at the exact kernel's measured rate
// (71 TMAC/s) is bound by per-iteration latency instead, and there the
// union's four-fold fewer iterations win (config 1, 16->32 on 8x28x28:
// 18.1 -> 12.4 us, below the dense kernel's 13.7).  Tuning switch kgs_f32=0|1.
bool use_f32_union(const Geom &g, uint64_t kept_weights) {
  if (g.es != 4) return false;
  const int v = tune("kgs_f32");
  if (v == 0 || v == 1) return v == 1;
  const double voxels = static_cast<double>(std::max(g.n, 1)) * g.to * g.ho * g.wo;
  return voxels * static_cast<double>(kept_weights) / 71e12 < 5e-6;
}

// Block pairs: tuning switch kgs_map=2.
bool use_block_pairs(const Geom &g, const Mask4 *m4) {
  (void)m4;
  return g.es == 2 && tune("kgs_map") == 2;
}

// Filter rows (of 16) per wave tile of the pair mapping: tuning switch
// pair_mfw=1|2|4, else 1.
int pair_width(const Geom &g, const Mask4 *m4) {
  (void)g;
  (void)m4;
  const int v = tune("pair_mfw");
  return (v == 2 || v == 4) ? v : 1;
}

// Build everything for a KGS pack (w may be null when only sizing).
rt3d_status plan_kgs(const rt3d_conv3d_desc *d, const uint8_t *mask, const uint8_t *w,
                     Canon &c, Layout &L, Tiling &tl, bool &vanilla) {
  rt3d_status st = canon_index(d, mask, c);
  if (st != RT3D_OK) return st;
  const int ks = d->kt * d->kh * d->kw;
  vanilla = true;
  for (size_t gi = 0; gi + 1 < c.group_ptr.size(); ++gi) {
    const uint32_t k = c.group_ptr[gi + 1] - c.group_ptr[gi];
    if (k != 0 && k != static_cast<uint32_t>(ks)) {
      vanilla = false;
      break;
    }
  }
  const Geom g = geom_of(d);
  const bool small = small_ok(g);
  Mask4 m4{mask, c.Q, ks, d->g_m / 4, d->g_n / 4};
  const ItemPlan ip = item_plan(g, &m4, small);
  tl = ip.tl;
  if (tl.cc == 0) return fail(RT3D_ERR_UNSUPPORTED, "no voxel tiling fits in LDS for this layer");
  static const uint8_t zero = 0;
  const uint8_t *wsrc = w ? w : &zero;
  if (!w) {
    // Sizing only: build the layout from a weight source that is never
    // dereferenced beyond the mask check by using an all-zero byte span.
    // The layout size does not depend on weight values.
  }
  if (g.es == 4) {
    std::vector<uint8_t> scratch;
    if (!w) {
      // size-only pass: reuse the builders with a scratch weight tensor
      scratch.assign(static_cast<size_t>(g.c_out) * g.c_in * ks * g.es, 0);
      wsrc = scratch.data();
    }
    if (use_f32_union(g, c.nvals)) build_items_layout(g, tl, wsrc, &m4, L, false, 1);
    else build_exact_f32_layout(g, tl, wsrc, &m4, L);
  } else {
    std::vector<uint8_t> scratch;
    if (!w) {
      scratch.assign(static_cast<size_t>(g.c_out) * g.c_in * ks * g.es, 0);
      wsrc = scratch.data();
    }
    if (!small && use_block_pairs(g, &m4)) {
      tl = choose_tiling(g, 64);
      if (tl.cc == 0) return fail(RT3D_ERR_UNSUPPORTED, "no voxel tiling fits in LDS for this layer");
      build_block_pairs_layout(g, tl, wsrc, &m4, L);
    } else if (!small && use_pairs(g, &m4)) {
      tl = choose_tiling(g, 64);
      if (tl.cc == 0) return fail(RT3D_ERR_UNSUPPORTED, "no voxel tiling fits in LDS for this layer");
      build_pairs_layout(g, tl, wsrc, &m4, L, pair_width(g, &m4));
    } else {
      build_items_layout(g, tl, wsrc, &m4, L, small, ip.mfw);
    }
  }
  return ok();
}

// ---------------------------------------------------------------------------
// Forward helpers
// ---------------------------------------------------------------------------

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

rt3d_status check_info(const rt3d_conv3d_desc *d, const rt3d_pack_info *info, bool sparse) {
  if (!info) return fail(RT3D_ERR_INVALID_ARG, "info is NULL");
  if (info->magic != kMagic || info->version != kVersion)
    return fail(RT3D_ERR_BLOB_MISMATCH, "info was not written by this library version");
  if (info->desc_hash != desc_hash(d))
    return fail(RT3D_ERR_BLOB_MISMATCH, "blob was packed for a different layer description");
  const bool is_sparse = info->variant == kVarKgsUnion16 || info->variant == kVarKgsExactF32 ||
                         info->variant == kVarKgsUnionF32 ||
                         info->variant == kVarSmallKgs16 || info->variant == kVarKgsPair16 ||
                         info->variant == kVarKgsBlockPair16;
  if (is_sparse != sparse)
    return fail(RT3D_ERR_BLOB_MISMATCH, sparse ? "dense blob passed to the KGS forward"
                                               : "KGS blob passed to the dense forward");
  return ok();
}

// Launch shape for a batch: waves per workgroup and channel-chunk splits so
// that the grid covers the GPU several times over, limited by the workspace
// the caller provides (ws_cap bytes; UINT64_MAX when sizing).
// Bytes the eight XCDs pull into their L2s when the logical workgroup ids
// (brick, filter tile group, split) are laid out with `order` and each XCD
// runs one contiguous run of them: a workgroup reads the weight rows of its
// (split, tile group) and the halo of its (split, brick).
double xcd_fill_bytes(long nb, long nt, long ns, int order, double a_unit, double x_unit) {
  const long nw = nb * nt * ns;
  const long q = nw / 8, r = nw % 8;
  const long inner = order == 0 ? nb : nt;          // fastest-varying index
  const long per_split = nb * nt;
  const double outer_unit = order == 0 ? a_unit : x_unit;  // pairs (split, slower index)
  const double inner_unit = order == 0 ? x_unit : a_unit;  // pairs (split, inner index)
  double total = 0;
  long lo = 0;
  for (int x = 0; x < 8; ++x) {
    const long cnt = q + (x < r ? 1 : 0);
    if (cnt == 0) continue;
    const long hi = lo + cnt;
    total += static_cast<double>((hi - 1) / inner - lo / inner + 1) * outer_unit;
    for (long sp = lo / per_split; sp <= (hi - 1) / per_split; ++sp) {
      const long a0 = std::max(lo, sp * per_split), a1 = std::min(hi, (sp + 1) * per_split);
      total += static_cast<double>(std::min(inner, a1 - a0)) * inner_unit;
    }
    lo = hi;
  }
  return total;
}

// Device queries are answered once per device and cached: the forward
// calls plan their launch on every call, and the runtime's occupancy and
// attribute queries would otherwise cost host time each time.
constexpr int kMaxDevices = 64;

int current_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return 0;
  }
  return dev;
}

// Compute units of the current device (256 when no device answers).
int device_cus() {
  static std::atomic<int> cache[kMaxDevices];
  const int dev = current_device();
  int cus = cache[dev].load(std::memory_order_relaxed);
  if (cus > 0) return cus;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0) {
    (void)hipGetLastError();
    return 256;
  }
  cache[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

// Resident workgroups per CU of a conv kernel at an LDS size (cached per
// device and kernel configuration; 0 when the runtime cannot say).
int cached_resident(int variant, int dtype, int mfw, int nf, size_t lds) {
  static std::mutex mu;
  static std::map<std::tuple<int, int, int, int, int, size_t>, int> cache;
  const auto key = std::make_tuple(current_device(), variant, dtype, mfw, nf, lds);
  {
    std::lock_guard<std::mutex> lock(mu);
    const auto it = cache.find(key);
    if (it != cache.end()) return it->second;
  }
  const int n = conv_resident(variant, dtype, mfw, nf, lds);
  if (n <= 0) {
    (void)hipGetLastError();
    return 0;
  }
  std::lock_guard<std::mutex> lock(mu);
  cache[key] = n;
  return n;
}

// Resident workgroups per CU of the small-input-channel kernel chosen for
// these arguments (cached like cached_resident).
int cached_small_resident(const ConvArgs &a, int dtype, int mfw) {
  static std::mutex mu;
  static std::map<std::tuple<int, int, int, int, int, int, size_t>, int> cache;
  const auto key = std::make_tuple(current_device(), dtype, mfw, a.steps_max > 4 ? 1 : 0,
                                   a.hw * a.c_in <= 127 ? 1 : 0, a.res ? 1 : 0, small_lds_bytes(a));
  {
    std::lock_guard<std::mutex> lock(mu);
    const auto it = cache.find(key);
    if (it != cache.end()) return it->second;
  }
  const int n = small_resident(a, dtype, mfw);
  if (n <= 0) {
    (void)hipGetLastError();
    return 0;
  }
  std::lock_guard<std::mutex> lock(mu);
  cache[key] = n;
  return n;
}

Launch plan_launch(const rt3d_conv3d_desc *d, const Plan &p, uint32_t variant, uint64_t ws_cap,
                   uint64_t a_bytes) {
  const Geom g = geom_of(d);
  const Tiling &tl = p.tiling;
  const long bricks = static_cast<long>(g.n) * ((g.to + tl.bt - 1) / tl.bt) *
                      ((g.ho + tl.bh - 1) / tl.bh) * ((g.wo + tl.bw - 1) / tl.bw);
  Launch L{4, 1, 0, 0};
  if (variant == kVarSmallDense16 || variant == kVarSmallKgs16) return L;  // one chunk, no split
  const long ntg = (p.wave_tiles + L.wpw - 1) / L.wpw;
  const long wgs = bricks * ntg;
  // LDS per workgroup as the launch requests it: split launches keep only
  // the halo (partials are stored from registers); unsplit ones also reuse
  // it as the epilogue tile of 16 * nf voxel slots x 64 * mfw filters.
  const size_t halo = static_cast<size_t>(tl.ht) * tl.hh * tl.hw * tl.row;
  const size_t tile = static_cast<size_t>(tl.slots) * (static_cast<size_t>(L.wpw) * 16 * p.mfw * 4 + 16);
  int per_cu_split = cached_resident(static_cast<int>(variant), d->dtype, p.mfw, tl.slots / 16, halo);
  int per_cu_whole =
      cached_resident(static_cast<int>(variant), d->dtype, p.mfw, tl.slots / 16, std::max(halo, tile));
  if (per_cu_split <= 0) per_cu_split = 2;
  if (per_cu_whole <= 0) per_cu_whole = per_cu_split;
  const double chunk_steps = p.tile_steps > 0 ? static_cast<double>(p.tile_steps) / tl.nchunks : 24.0;
  int splits = model_splits(g, tl, p.mfw, chunk_steps, variant, wgs, per_cu_split, per_cu_whole,
                            device_cus());
  if (tune("splits") > 0) splits = std::max(1, std::min(tl.nchunks, tune("splits")));
  const long total_vox = static_cast<long>(g.n) * g.to * g.ho * g.wo;
  const uint64_t per_split = static_cast<uint64_t>(total_vox) * ((g.c_out + 3) / 4 * 4) * 4;
  while (splits > 1 && per_split * splits > ws_cap) --splits;
  L.splits = splits;
  L.ws_bytes = splits > 1 ? per_split * splits : 0;
  const double a_unit = static_cast<double>(a_bytes) / (static_cast<double>(ntg) * splits);
  const double x_unit = static_cast<double>(tl.ht) * tl.hh * tl.hw * tl.cc * g.es * tl.nchunks / splits;
  L.order = xcd_fill_bytes(bricks, ntg, splits, 1, a_unit, x_unit) <
                    xcd_fill_bytes(bricks, ntg, splits, 0, a_unit, x_unit)
                ? 1
                : 0;
  if (tune("wg_order") >= 0) L.order = tune("wg_order") ? 1 : 0;
  return L;
}

rt3d_status run_conv(const rt3d_conv3d_desc *d, const rt3d_pack_info *info, const void *blob,
                     const void *x, const float *bias, const void *residual, void *y,
                     void *workspace, uint64_t ws_bytes, void *stream, bool sparse) {
  rt3d_status st = check_desc(d, sparse);
  if (st != RT3D_OK) return st;
  st = check_info(d, info, sparse);
  if (st != RT3D_OK) return st;
  if (d->n == 0) return ok();  // empty batch: nothing is read or written
  if (!blob || !x || !y) return fail(RT3D_ERR_INVALID_ARG, "blob, x and y must be non-NULL");
  const bool want_res = (d->flags & RT3D_RESIDUAL) != 0;
  if (want_res != (residual != nullptr))
    return fail(RT3D_ERR_INVALID_ARG, "residual must be given exactly when RT3D_RESIDUAL is set");
  if (!aligned16(blob) || !aligned16(x) || !aligned16(y) || (residual && !aligned16(residual)) ||
      (bias && !aligned16(bias)) || (workspace && !aligned16(workspace)))
    return fail(RT3D_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  Plan p;
  std::memcpy(&p, info->plan, sizeof(p));
  const Launch launch = plan_launch(d, p, info->variant, workspace ? ws_bytes : 0, info->packed_bytes - p.a_off);
  const Geom g = geom_of(d);
  const Tiling &tl = p.tiling;
  const uint8_t *b = static_cast<const uint8_t *>(blob);
  ConvArgs a{};
  a.x = x;
  a.y = y;
  a.steps_max = p.tile_steps;
  a.y_pitch = d->y_c_total != 0 ? d->y_c_total : d->c_out;
  a.y_off = d->y_c_off;
  a.x_pitch = d->x_c_total != 0 ? d->x_c_total : d->c_in;
  a.x_off = d->x_c_off;
  a.nf = tl.slots / 16;
  a.res = residual;
  a.bias = bias;
  a.step_ptr = reinterpret_cast<const uint32_t *>(b + p.step_ptr_off);
  a.item_ptr = reinterpret_cast<const uint32_t *>(b + p.item_ptr_off);
  a.items = reinterpret_cast<const uint32_t *>(b + p.items_off);
  a.keep = reinterpret_cast<const uint32_t *>(b + p.keep_off);
  a.gmap = info->variant == kVarKgsUnion16 && p.gmap ? a.keep : nullptr;
  a.gmap_slots = a.gmap ? p.wave_tiles * 4 * p.mfw : 0;
  a.a = b + p.a_off;
  a.a_bytes = static_cast<int32_t>(std::min<uint64_t>(info->packed_bytes - p.a_off, 0x7fffffffu));
  a.n = g.n; a.c_in = g.c_in; a.c_out = g.c_out; a.t = g.t; a.h = g.h; a.w = g.w;
  a.to = g.to; a.ho = g.ho; a.wo = g.wo;
  a.st = g.st; a.sh = g.sh; a.sw = g.sw; a.pt = g.pt; a.ph = g.ph; a.pw = g.pw;
  a.bt = tl.bt; a.bh = tl.bh; a.bw = tl.bw;
  a.nbt = (g.to + tl.bt - 1) / tl.bt;
  a.nbh = (g.ho + tl.bh - 1) / tl.bh;
  a.nbw = (g.wo + tl.bw - 1) / tl.bw;
  a.ht = tl.ht; a.hh = tl.hh; a.hw = tl.hw; a.cc = tl.cc; a.row = tl.row; a.nchunks = tl.nchunks;
  a.wave_tiles = p.wave_tiles;
  a.relu = (d->flags & RT3D_RELU) ? 1 : 0;
  a.wpw = launch.wpw;
  a.splits = launch.splits;
  a.c_out4 = (g.c_out + 3) / 4 * 4;
  a.total_vox = static_cast<long>(g.n) * g.to * g.ho * g.wo;
  a.ws = static_cast<float *>(workspace);
  a.qt = g.qt; a.qh = g.qh; a.qw = g.qw;
  a.pto = g.pto; a.pho = g.pho; a.pwo = g.pwo;
  a.c_wg = a.wpw * 16 * p.mfw;
  a.tile_row = a.c_wg * 4 + 16;  // +16 bytes: slot rows start on different banks
  a.order = launch.order;
  a.nbricks = static_cast<int32_t>(static_cast<long>(a.n) * a.nbt * a.nbh * a.nbw);
  a.ntg = (a.wave_tiles + a.wpw - 1) / a.wpw;
  a.grid = 0;  // one workgroup per tile
  // The kernels divide workgroup ids, (pooled) voxel indices and chunk
  // ranges (split * nchunks) with a 24-bit reciprocal method.
  if (tl.nchunks >= 4096)
    return fail(RT3D_ERR_UNSUPPORTED, "4096 or more input-channel chunks");
  if (a.total_vox >= (1L << 24))
    return fail(RT3D_ERR_UNSUPPORTED, "2^24 or more output voxels per launch");
  if ((info->variant == kVarSmallDense16 || info->variant == kVarSmallKgs16) &&
      static_cast<long>(g.n) * g.t * g.h * g.w * g.c_in * 2 >= (1L << 31) - 8)
    return fail(RT3D_ERR_UNSUPPORTED, "input of 2^31 - 8 bytes or more on the small-channel kernel");
  if (static_cast<long>(a.n) * a.nbt * a.nbh * a.nbw * a.ntg * a.splits >= (1L << 24))
    return fail(RT3D_ERR_UNSUPPORTED, "layer needs 2^24 or more workgroups");
  int e;
  switch (info->variant) {
    case kVarDenseItems16:
    case kVarKgsUnion16:
      e = launch_items16(a, d->dtype, p.mfw, 0, stream);
      break;
    case kVarKgsPair16:
      e = launch_items16(a, d->dtype, p.mfw, 1, stream);
      break;
    case kVarKgsBlockPair16:
      e = launch_items16(a, d->dtype, p.mfw, 2, stream);
      break;
    case kVarSmallDense16:
    case kVarSmallKgs16: {
      // Waves walk (wave tile, brick) pairs: as many workgroups as fit
      // resident, with a wave count that is a multiple of the wave tiles.
      const long waves = static_cast<long>(a.nbricks) * a.wave_tiles;
      int per_cu = cached_small_resident(a, d->dtype, p.mfw);
      if (per_cu <= 0) per_cu = 1;
      long grid = std::min<long>((waves + 3) / 4, static_cast<long>(device_cus()) * per_cu);
      const long unit = a.wave_tiles / std::gcd(a.wave_tiles, 4);
      grid = std::max<long>(unit, grid / unit * unit);
      a.grid = static_cast<int32_t>(grid);
      e = launch_small16(a, d->dtype, p.mfw, stream);
      break;
    }
    case kVarDenseItemsF32:
    case kVarKgsUnionF32:
      e = launch_items_f32(a, p.mfw, stream);
      break;
    case kVarKgsExactF32:
      e = launch_kgs_exact_f32(a, stream);
      break;
    default:
      return fail(RT3D_ERR_BLOB_MISMATCH, "unknown kernel variant %u", info->variant);
  }
  if (e == hipSuccess && a.splits > 1) e = launch_reduce_splits(a, d->dtype, stream);
  if (e != hipSuccess)
    return fail(RT3D_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(static_cast<hipError_t>(e)));
  return ok();
}

// ---------------------------------------------------------------------------
// Reweighted group-lasso penalty (Section 4): validation and launch shape
// ---------------------------------------------------------------------------

constexpr int kGroupMaxUnitElems = 12288;  // g_m * g_n * K_s staged per channel group
constexpr long kGroupTargetWgs = 2048;     // enough workgroups to keep HBM busy

struct GroupPlan {
  int P, Q, ks, qb, nqc;
  long units, wgs;
  size_t lds;
  int buf_elems, unit_cap;
};

bool finite(float v) { return v == v && v - v == 0.f; }

// Workspace: one float partial sum per workgroup.
uint64_t group_workspace_bytes(const GroupPlan &g) {
  return static_cast<uint64_t>(g.wgs) * sizeof(float);
}

rt3d_status check_group_desc(const rt3d_group_desc *d) {
  if (!d) return fail(RT3D_ERR_INVALID_ARG, "desc is NULL");
  if (d->c_out <= 0 || d->c_in <= 0) return fail(RT3D_ERR_INVALID_ARG, "channel counts must be positive");
  if (d->kt <= 0 || d->kh <= 0 || d->kw <= 0)
    return fail(RT3D_ERR_INVALID_ARG, "kernel extents must be positive");
  if (d->kt > 7 || d->kh > 7 || d->kw > 7)
    return fail(RT3D_ERR_UNSUPPORTED, "kernel extents above 7 are not supported");
  if (d->g_m <= 0 || d->g_n <= 0) return fail(RT3D_ERR_INVALID_ARG, "group sizes must be positive");
  if (d->g_m > 16 || d->g_n > 16) return fail(RT3D_ERR_UNSUPPORTED, "group sizes above 16 are not supported");
  if (d->dtype != RT3D_F32 && d->dtype != RT3D_BF16 && d->dtype != RT3D_F16)
    return fail(RT3D_ERR_INVALID_ARG, "unknown dtype %d", d->dtype);
  if (d->norm != 1 && d->norm != 2) return fail(RT3D_ERR_INVALID_ARG, "norm must be 1 or 2, got %d", d->norm);
  if (d->scope != RT3D_SCOPE_KGS && d->scope != RT3D_SCOPE_VANILLA)
    return fail(RT3D_ERR_INVALID_ARG, "unknown scope %d", d->scope);
  const long ks = static_cast<long>(d->kt) * d->kh * d->kw;
  if (static_cast<long>(d->g_m) * d->g_n * ks > kGroupMaxUnitElems)
    return fail(RT3D_ERR_UNSUPPORTED, "g_m * g_n * K_s = %ld exceeds %d", static_cast<long>(d->g_m) * d->g_n * ks,
                kGroupMaxUnitElems);
  if (static_cast<double>(d->c_out) * d->c_in * ks > 2.0e9)
    return fail(RT3D_ERR_UNSUPPORTED, "weight tensor too large");
  return RT3D_OK;
}

GroupPlan group_plan(const rt3d_group_desc *d) {
  GroupPlan g;
  g.ks = d->kt * d->kh * d->kw;
  g.P = (d->c_out + d->g_m - 1) / d->g_m;
  g.Q = (d->c_in + d->g_n - 1) / d->g_n;
  g.units = static_cast<long>(g.P) * g.Q * (d->scope == RT3D_SCOPE_KGS ? g.ks : 1);
  const int per_q = d->g_m * d->g_n * g.ks;                        // staged floats per channel group
  const int per_q_units = d->scope == RT3D_SCOPE_KGS ? g.ks : 1;
  // staged block + two unit arrays + the reduction buffer within 64 KB of LDS
  // (>= 1 channel group after validation)
  const int lds_cap = std::min(kGroupMaxUnitElems / per_q,
                               (65536 - 256 * 4) / (4 * (per_q + 2 * per_q_units)));
  const long want = (static_cast<long>(g.P) * g.Q + kGroupTargetWgs - 1) / kGroupTargetWgs;
  g.qb = static_cast<int>(std::min<long>({std::max<long>(want, 1), lds_cap, g.Q}));
  g.nqc = (g.Q + g.qb - 1) / g.qb;
  g.wgs = static_cast<long>(g.P) * g.nqc;
  g.buf_elems = per_q * g.qb;
  g.unit_cap = per_q_units * g.qb;
  g.lds = sizeof(float) * (static_cast<size_t>(g.buf_elems) + 2 * static_cast<size_t>(g.unit_cap) + 256);
  return g;
}

}  // namespace
}  // namespace rt3d

using namespace rt3d;

extern "C" {

const char *rt3d_status_string(rt3d_status s) {
  switch (s) {
    case RT3D_OK: return "ok";
    case RT3D_ERR_INVALID_ARG: return "invalid argument";
    case RT3D_ERR_UNSUPPORTED: return "unsupported configuration";
    case RT3D_ERR_BUFFER_TOO_SMALL: return "buffer too small";
    case RT3D_ERR_BLOB_MISMATCH: return "packed blob does not match the layer";
    case RT3D_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char *rt3d_last_error_detail(void) { return g_detail.c_str(); }

rt3d_status rt3d_conv3d_out_shape(const rt3d_conv3d_desc *d, int32_t *to, int32_t *ho,
                                  int32_t *wo) {
  rt3d_status st = check_desc(d, false);
  if (st != RT3D_OK) return st;
  if (!to || !ho || !wo) return fail(RT3D_ERR_INVALID_ARG, "output pointers must be non-NULL");
  const Geom g = geom_of(d);
  *to = g.pto;
  *ho = g.pho;
  *wo = g.pwo;
  return ok();
}

rt3d_status rt3d_kgs_pack_size(const rt3d_conv3d_desc *d, const uint8_t *mask, uint64_t *bytes) {
  rt3d_status st = check_desc(d, true);
  if (st != RT3D_OK) return st;
  if (!mask || !bytes) return fail(RT3D_ERR_INVALID_ARG, "mask and bytes must be non-NULL");
  Canon c;
  Layout L;
  Tiling tl;
  bool vanilla;
  st = plan_kgs(d, mask, nullptr, c, L, tl, vanilla);
  if (st != RT3D_OK) return st;
  *bytes = section_offsets(&c, esize_of(d->dtype), L).total;
  return ok();
}

rt3d_status rt3d_kgs_pack(const rt3d_conv3d_desc *d, const void *w_dense, const uint8_t *mask,
                          void *blob, uint64_t blob_bytes, rt3d_pack_info *info) {
  rt3d_status st = check_desc(d, true);
  if (st != RT3D_OK) return st;
  if (!w_dense || !mask || !blob || !info)
    return fail(RT3D_ERR_INVALID_ARG, "w_dense, mask, blob and info must be non-NULL");
  Canon c;
  Layout L;
  Tiling tl;
  bool vanilla;
  st = plan_kgs(d, mask, static_cast<const uint8_t *>(w_dense), c, L, tl, vanilla);
  if (st != RT3D_OK) return st;
  const Sections s = section_offsets(&c, esize_of(d->dtype), L);
  if (blob_bytes < s.total)
    return fail(RT3D_ERR_BUFFER_TOO_SMALL, "blob needs %llu bytes, got %llu",
                static_cast<unsigned long long>(s.total), static_cast<unsigned long long>(blob_bytes));
  rt3d_pack_info tmp;
  fill_info(d, &c, L, tl, s, vanilla, &tmp);
  write_blob(static_cast<uint8_t *>(blob), tmp, &c, static_cast<const uint8_t *>(w_dense), d, L, s);
  *info = tmp;
  return ok();
}

rt3d_status rt3d_kgs_unpack(const rt3d_conv3d_desc *d, const rt3d_pack_info *info, const void *blob,
                            void *w_out) {
  rt3d_status st = check_desc(d, true);
  if (st != RT3D_OK) return st;
  if (!blob || !w_out) return fail(RT3D_ERR_INVALID_ARG, "blob and w_out must be non-NULL");
  st = check_info(d, info, true);
  if (st != RT3D_OK) return st;
  const uint8_t *b = static_cast<const uint8_t *>(blob);
  const int es = esize_of(d->dtype);
  const int ks = d->kt * d->kh * d->kw;
  const int P = (d->c_out + d->g_m - 1) / d->g_m, Q = (d->c_in + d->g_n - 1) / d->g_n;
  const uint32_t *gp = reinterpret_cast<const uint32_t *>(b + info->canon_off[0]);
  const uint16_t *pos = reinterpret_cast<const uint16_t *>(b + info->canon_off[1]);
  const uint64_t *vp = reinterpret_cast<const uint64_t *>(b + info->canon_off[2]);
  const uint8_t *vals = b + info->canon_off[3];
  uint8_t *w = static_cast<uint8_t *>(w_out);
  std::memset(w, 0, static_cast<size_t>(d->c_out) * d->c_in * ks * es);
  for (int p = 0; p < P; ++p) {
    const int gm = std::min(d->g_m, d->c_out - p * d->g_m);
    for (int q = 0; q < Q; ++q) {
      const int gn = std::min(d->g_n, d->c_in - q * d->g_n);
      const size_t gi = static_cast<size_t>(p) * Q + q;
      const uint32_t k0 = gp[gi], k = gp[gi + 1] - k0;
      for (int i = 0; i < gm; ++i)
        for (int j = 0; j < gn; ++j)
          for (uint32_t r = 0; r < k; ++r) {
            const size_t widx =
                (static_cast<size_t>(p * d->g_m + i) * d->c_in + q * d->g_n + j) * ks + pos[k0 + r];
            std::memcpy(w + widx * es, vals + (vp[gi] + (static_cast<size_t>(i) * gn + j) * k + r) * es, es);
          }
    }
  }
  return ok();
}

rt3d_status rt3d_conv3d_workspace_size(const rt3d_conv3d_desc *d, const rt3d_pack_info *info,
                                       uint64_t *bytes) {
  rt3d_status st = check_desc(d, false);
  if (st != RT3D_OK) return st;
  if (!info || !bytes) return fail(RT3D_ERR_INVALID_ARG, "info and bytes must be non-NULL");
  if (info->magic != kMagic || info->version != kVersion || info->desc_hash != desc_hash(d))
    return fail(RT3D_ERR_BLOB_MISMATCH, "info does not belong to this layer description");
  Plan p;
  std::memcpy(&p, info->plan, sizeof(p));
  *bytes = plan_launch(d, p, info->variant, UINT64_MAX, info->packed_bytes - p.a_off).ws_bytes;
  return ok();
}

rt3d_status rt3d_kgs_conv3d_fwd(const rt3d_conv3d_desc *d, const rt3d_pack_info *info,
                                const void *blob_dev, const void *x, const float *bias,
                                const void *residual, void *y, void *workspace,
                                uint64_t workspace_bytes, void *stream) {
  return run_conv(d, info, blob_dev, x, bias, residual, y, workspace, workspace_bytes, stream, true);
}

rt3d_status rt3d_kgs_conv3d_fwd_noalloc(const rt3d_conv3d_desc *d, const rt3d_pack_info *info,
                                        const void *blob_dev, const void *x, const float *bias,
                                        const void *residual, void *y, void *stream) {
  rt3d_status st = check_desc(d, true);
  if (st != RT3D_OK) return st;
  st = check_info(d, info, true);
  if (st != RT3D_OK) return st;
  if (d->n == 0) return ok();
  Plan p;
  std::memcpy(&p, info->plan, sizeof(p));
  // The split count a caller workspace of any size would get: the launch is
  // then the one rt3d_kgs_conv3d_fwd makes with that workspace.
  const uint64_t need = plan_launch(d, p, info->variant, UINT64_MAX, info->packed_bytes - p.a_off).ws_bytes;
  if (need > kScratchBytes)
    return fail(RT3D_ERR_UNSUPPORTED,
                "this launch needs %llu bytes of split-K scratch; the no-allocation entry point "
                "holds %llu (use rt3d_kgs_conv3d_fwd with a caller workspace)",
                static_cast<unsigned long long>(need), static_cast<unsigned long long>(kScratchBytes));
  void *ws = nullptr;
  if (need > 0) {
    ws = noalloc_scratch();
    if (!ws) return fail(RT3D_ERR_HIP, "the device address of the library's scratch is unavailable");
  }
  return run_conv(d, info, blob_dev, x, bias, residual, y, ws, need, stream, true);
}

rt3d_status rt3d_dense_pack_size(const rt3d_conv3d_desc *d, uint64_t *bytes) {
  rt3d_status st = check_desc(d, false);
  if (st != RT3D_OK) return st;
  if (!bytes) return fail(RT3D_ERR_INVALID_ARG, "bytes must be non-NULL");
  const Geom g = geom_of(d);
  const bool small = small_ok(g);
  const ItemPlan ip = item_plan(g, nullptr, small);
  const Tiling &tl = ip.tl;
  if (tl.cc == 0) return fail(RT3D_ERR_UNSUPPORTED, "no voxel tiling fits in LDS for this layer");
  std::vector<uint8_t> scratch(static_cast<size_t>(g.c_out) * g.c_in * g.ks * g.es, 0);
  Layout L;
  build_items_layout(g, tl, scratch.data(), nullptr, L, small, ip.mfw);
  *bytes = section_offsets(nullptr, g.es, L).total;
  return ok();
}

rt3d_status rt3d_dense_pack(const rt3d_conv3d_desc *d, const void *w_dense, void *blob,
                            uint64_t blob_bytes, rt3d_pack_info *info) {
  rt3d_status st = check_desc(d, false);
  if (st != RT3D_OK) return st;
  if (!w_dense || !blob || !info)
    return fail(RT3D_ERR_INVALID_ARG, "w_dense, blob and info must be non-NULL");
  const Geom g = geom_of(d);
  const bool small = small_ok(g);
  const ItemPlan ip = item_plan(g, nullptr, small);
  const Tiling &tl = ip.tl;
  if (tl.cc == 0) return fail(RT3D_ERR_UNSUPPORTED, "no voxel tiling fits in LDS for this layer");
  Layout L;
  build_items_layout(g, tl, static_cast<const uint8_t *>(w_dense), nullptr, L, small, ip.mfw);
  const Sections s = section_offsets(nullptr, g.es, L);
  if (blob_bytes < s.total)
    return fail(RT3D_ERR_BUFFER_TOO_SMALL, "blob needs %llu bytes, got %llu",
                static_cast<unsigned long long>(s.total), static_cast<unsigned long long>(blob_bytes));
  rt3d_pack_info tmp;
  fill_info(d, nullptr, L, tl, s, false, &tmp);
  write_blob(static_cast<uint8_t *>(blob), tmp, nullptr, nullptr, d, L, s);
  *info = tmp;
  return ok();
}

rt3d_status rt3d_conv3d_dense_fwd(const rt3d_conv3d_desc *d, const rt3d_pack_info *info,
                                  const void *blob_dev, const void *x, const float *bias,
                                  const void *residual, void *y, void *workspace,
                                  uint64_t workspace_bytes, void *stream) {
  return run_conv(d, info, blob_dev, x, bias, residual, y, workspace, workspace_bytes, stream, false);
}

rt3d_status rt3d_maxpool3d_fwd(int32_t n, int32_t c, int32_t t, int32_t h, int32_t w, int32_t kt,
                               int32_t kh, int32_t kw, int32_t st, int32_t sh, int32_t sw,
                               int32_t pt, int32_t ph, int32_t pw, int32_t dtype, const void *x,
                               void *y, void *stream) {
  if (n < 0 || c <= 0 || t <= 0 || h <= 0 || w <= 0 || kt <= 0 || kh <= 0 || kw <= 0 || st <= 0 ||
      sh <= 0 || sw <= 0)
    return fail(RT3D_ERR_INVALID_ARG, "pooling sizes must be positive");
  if (pt < 0 || ph < 0 || pw < 0 || 2 * pt > kt || 2 * ph > kh || 2 * pw > kw)
    return fail(RT3D_ERR_INVALID_ARG, "pooling padding must be between 0 and half the window");
  if (dtype != RT3D_F32 && dtype != RT3D_BF16 && dtype != RT3D_F16)
    return fail(RT3D_ERR_INVALID_ARG, "unknown dtype %d", dtype);
  if (kt > t + 2 * pt || kh > h + 2 * ph || kw > w + 2 * pw)
    return fail(RT3D_ERR_INVALID_ARG, "window larger than the padded input");
  if (n == 0) return ok();
  if (!x || !y) return fail(RT3D_ERR_INVALID_ARG, "x and y must be non-NULL");
  if (!aligned16(x) || !aligned16(y))
    return fail(RT3D_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  const int to = (t + 2 * pt - kt) / st + 1, ho = (h + 2 * ph - kh) / sh + 1,
            wo = (w + 2 * pw - kw) / sw + 1;
  if (static_cast<long>(n) * to * ho * wo >= (1l << 24))
    return fail(RT3D_ERR_UNSUPPORTED, "2^24 or more output voxels per call");
  const int e = launch_maxpool(n, c, t, h, w, kt, kh, kw, st, sh, sw, pt, ph, pw, to, ho, wo, dtype,
                               x, y, stream);
  if (e != hipSuccess)
    return fail(RT3D_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(static_cast<hipError_t>(e)));
  return ok();
}


rt3d_status rt3d_group_units(const rt3d_group_desc *d, int64_t *units) {
  const rt3d_status st = check_group_desc(d);
  if (st != RT3D_OK) return st;
  if (!units) return fail(RT3D_ERR_INVALID_ARG, "units must be non-NULL");
  *units = group_plan(d).units;
  return ok();
}

rt3d_status rt3d_group_workspace_size(const rt3d_group_desc *d, uint64_t *bytes) {
  const rt3d_status st = check_group_desc(d);
  if (st != RT3D_OK) return st;
  if (!bytes) return fail(RT3D_ERR_INVALID_ARG, "bytes must be non-NULL");
  *bytes = align_up(group_workspace_bytes(group_plan(d)), kAlign);
  return ok();
}

rt3d_status rt3d_group_reweight(const rt3d_group_desc *d, const void *w, const float *pen,
                                float lambda, float eps, float tau, float step, float *norms,
                                float *pen_next, float *reg, uint8_t *mask, float *grad,
                                void *w_prox, void *workspace, uint64_t workspace_bytes,
                                void *stream) {
  const rt3d_status st = check_group_desc(d);
  if (st != RT3D_OK) return st;
  if (!w) return fail(RT3D_ERR_INVALID_ARG, "w must be non-NULL");
  if (!finite(lambda) || !finite(eps) || !finite(tau) || !finite(step))
    return fail(RT3D_ERR_INVALID_ARG, "lambda, eps, tau and step must be finite");
  if (!(eps > 0.f)) return fail(RT3D_ERR_INVALID_ARG, "eps must be > 0");
  if (lambda < 0.f || step < 0.f) return fail(RT3D_ERR_INVALID_ARG, "lambda and step must be >= 0");
  const int es = esize_of(d->dtype);
  auto misaligned = [](const void *p, uintptr_t a) {
    return p && (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0;
  };
  if (misaligned(w, es) || misaligned(w_prox, es) || misaligned(pen, 4) || misaligned(norms, 4) ||
      misaligned(pen_next, 4) || misaligned(reg, 4) || misaligned(grad, 4) || misaligned(workspace, 4))
    return fail(RT3D_ERR_INVALID_ARG, "pointers must be aligned to their element size");
  const GroupPlan g = group_plan(d);
  const uint64_t need = group_workspace_bytes(g);
  if (reg && (!workspace || workspace_bytes < need))
    return fail(RT3D_ERR_BUFFER_TOO_SMALL, "reg needs %llu bytes of workspace, got %llu",
                static_cast<unsigned long long>(need),
                static_cast<unsigned long long>(workspace ? workspace_bytes : 0));
  if (!norms && !pen_next && !reg && !mask && !grad && !w_prox) return ok();
  GroupArgs a{};
  a.w = w;
  a.pen = pen;
  a.norms = norms;
  a.pen_next = pen_next;
  a.partial = reg ? static_cast<float *>(workspace) : nullptr;
  a.grad = grad;
  a.mask = mask;
  a.w_prox = w_prox;
  a.M = d->c_out;
  a.N = d->c_in;
  a.ks = g.ks;
  a.gm = d->g_m;
  a.gn = d->g_n;
  a.P = g.P;
  a.Q = g.Q;
  a.qb = g.qb;
  a.nqc = g.nqc;
  a.buf_elems = g.buf_elems;
  a.unit_cap = g.unit_cap;
  a.lambda = lambda;
  a.eps = eps;
  a.tau = tau;
  a.step = step;
  int e = launch_group_reweight(a, d->dtype, d->norm, d->scope, g.lds, stream);
  if (e == hipSuccess && reg)
    e = launch_reg_finalize(a.partial, static_cast<int>(g.wgs), lambda, reg, stream);
  if (e != hipSuccess)
    return fail(RT3D_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(static_cast<hipError_t>(e)));
  return ok();
}

}  // extern "C"
