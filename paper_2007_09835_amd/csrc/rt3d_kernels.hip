// HIP kernels of librt3d for gfx950 (MI355X): forward 3-D convolution, dense
// and kernel-group-structured (KGS) sparse, plus 3-D max pooling.
//
// Structure shared by the conv kernels (paper: RT3D, arXiv 2007.09835).  A
// KGS layer equals the dense layer with whole columns removed from each
// kernel group's g_M x (g_N*K_s) matrix (Section 3, reshaping paragraph),
// so after packing every group is a dense contraction.  Here the columns
// are "items": one 4-channel block at one kernel position.  A workgroup
// owns a brick of output voxels of one batch item; for each chunk of input
// channels it stages the input brick plus halo in LDS (coalesced 16-byte
// loads along the channel axis, zero fill for padding and missing channels),
// then walks the items it must multiply.  An item's operand is the staged
// brick read at a constant shift (the kernel position) and channel offset,
// so the implicit-GEMM gather costs one LDS address add per item.
//
// Tensors are channels-last: x [n][t][h][w][c_in], y [n][to][ho][wo][c_out].

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <mutex>

#include <type_traits>
#include <utility>

#include "rt3d_internal.h"

namespace rt3d {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(16 * sizeof(__bf16)))) __bf16 bf16x16;
typedef __attribute__((__vector_size__(16 * sizeof(_Float16)))) _Float16 f16x16;
typedef __attribute__((__vector_size__(8 * sizeof(unsigned)))) unsigned u32x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(unsigned)))) unsigned u32x4;

template <int... Is, typename F>
__device__ __forceinline__ void static_for_impl(std::integer_sequence<int, Is...>, F &&f) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
  static_for_impl(std::make_integer_sequence<int, N>{}, f);
}

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ uint32_t uniform(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(v)));
}

// n / d and n % d for 0 <= n < 2^24 and 1 <= d < 2^24.  The fp32 reciprocal
// estimate has relative error below 2^-22, so for quotients below 2^21 the
// truncated product is off by at most one, which one step corrects.  (The
// host keeps every index divided here below 2^24.)
struct DivMod {
  int q, r;
};

__device__ __forceinline__ DivMod divmod(int n, int d) {
  int q = static_cast<int>(static_cast<float>(n) * __builtin_amdgcn_rcpf(static_cast<float>(d)));
  const int r0 = n - q * d;
  const int fix = (r0 >= d ? 1 : 0) - (r0 < 0 ? 1 : 0);  // selects, no branches
  q += fix;
  return {q, r0 - fix * d};
}

// ---------------------------------------------------------------------------
// Brick geometry
// ---------------------------------------------------------------------------

struct Brick {
  int nb;               // batch item
  int ot0, oh0, ow0;    // first output voxel of the brick
  int zt0, zh0, zw0;    // input coordinate of halo voxel (0, 0, 0)
};

// Workgroup coordinates.  The hardware hands consecutive workgroup ids to
// the eight XCDs in turn (id mod 8); remapping so that each XCD receives one
// contiguous run of logical ids keeps the workgroups that share weight rows
// (order 0: bricks fastest) or halo bricks (order 1: filter tiles fastest) in
// one XCD's L2.  The remap is a bijection for any grid size.
struct Wg {
  int brick, tg, split;
};

// Logical tile id -> (brick, filter tile group, split).
__device__ __forceinline__ Wg decode_tile(const ConvArgs &a, int lid) {
  Wg g;
  if (a.order == 0) {
    const DivMod x = divmod(lid, a.nbricks), y = divmod(x.q, a.ntg);
    g.brick = x.r;
    g.tg = y.r;
    g.split = y.q;
  } else {
    const DivMod x = divmod(lid, a.ntg), y = divmod(x.q, a.nbricks);
    g.tg = x.r;
    g.brick = y.r;
    g.split = y.q;
  }
  g.brick = uniform(g.brick);
  g.tg = uniform(g.tg);
  g.split = uniform(g.split);
  return g;
}

// Logical id of this workgroup's tile in a one-tile-per-workgroup grid.
__device__ __forceinline__ int xcd_remap(int nw) {
  const int id = static_cast<int>(blockIdx.x);
  const int q = nw >> 3, r = nw & 7;
  const int xcd = id & 7, local = id >> 3;
  return xcd < r ? xcd * (q + 1) + local : r * (q + 1) + (xcd - r) * q + local;
}

__device__ __forceinline__ Wg decode_wg(const ConvArgs &a) {
  return decode_tile(a, xcd_remap(a.nbricks * a.ntg * a.splits));
}

__device__ __forceinline__ Brick decode_brick(const ConvArgs &a, int brick) {
  Brick b;
  const DivMod x = divmod(brick, a.nbw), y = divmod(x.q, a.nbh), z = divmod(y.q, a.nbt);
  const int bwi = x.r, bhi = y.r, bti = z.r;
  b.nb = z.q;
  b.ot0 = bti * a.bt;
  b.oh0 = bhi * a.bh;
  b.ow0 = bwi * a.bw;
  b.zt0 = b.ot0 * a.st - a.pt;
  b.zh0 = b.oh0 * a.sh - a.ph;
  b.zw0 = b.ow0 * a.sw - a.pw;
  return b;
}

// Voxel slot s of the brick: LDS byte offset of its (0,0,0) kernel tap in
// the halo, flat index of its output voxel, and whether it exists.
struct Slot {
  int lds;
  long out;
  bool valid;
};

__device__ __forceinline__ Slot slot_at(const ConvArgs &a, const Brick &b, int tt, int hh, int ww) {
  Slot o;
  o.valid = tt < a.bt && b.ot0 + tt < a.to && b.oh0 + hh < a.ho && b.ow0 + ww < a.wo;
  if (!o.valid) tt = hh = ww = 0;
  o.lds = (((tt * a.st) * a.hh + hh * a.sh) * a.hw + ww * a.sw) * a.row;
  o.out = ((static_cast<long>(b.nb) * a.to + b.ot0 + tt) * a.ho + b.oh0 + hh) * a.wo + b.ow0 + ww;
  return o;
}

// LDS byte offset of voxel slot (tt, hh, ww)'s (0,0,0) tap: the part of
// slot_at the K loop needs, without branches.  Slots outside the output read
// slot 0's row (their results are never stored).
__device__ __forceinline__ int slot_lds(const ConvArgs &a, const Brick &b, int tt, int hh, int ww) {
  const bool valid = (tt < a.bt) & (b.ot0 + tt < a.to) & (b.oh0 + hh < a.ho) & (b.ow0 + ww < a.wo);
  tt = valid ? tt : 0;
  hh = valid ? hh : 0;
  ww = valid ? ww : 0;
  return (((tt * a.st) * a.hh + hh * a.sh) * a.hw + ww * a.sw) * a.row;
}

// (t, h, w) of voxel slots s, s + stride, s + 2*stride, ... of the brick:
// one divmod pair to start, then carries only (VALU time in the prologue
// and epilogue is otherwise dominated by divisions).
struct SlotWalk {
  int t, h, w, dt, dh, dw;
  __device__ __forceinline__ void init(const ConvArgs &a, int s, int stride) {
    const int plane = a.bh * a.bw;
    const DivMod x = divmod(s, plane), y = divmod(x.r, a.bw);
    t = x.q;
    h = y.q;
    w = y.r;
    const DivMod p = divmod(stride, plane), q = divmod(p.r, a.bw);
    dt = p.q;
    dh = q.q;
    dw = q.r;
  }
  __device__ __forceinline__ void next(const ConvArgs &a) {
    w += dw;
    const int cw = w >= a.bw ? 1 : 0;
    w -= cw * a.bw;
    h += dh + cw;
    const int chh = h >= a.bh ? 1 : 0;
    h -= chh * a.bh;
    t += dt + chh;
  }
};

// Stage channels [c0, c0 + cc) of the input brick plus halo into LDS.
// Row r of the halo (one input voxel) holds cc channels, zero where the
// voxel is padding or the channel does not exist.
// ILV (16-bit block-pair mapping): each 16-byte piece of 8 channels -- the
// 4-channel blocks 2i and 2i + 1 -- is stored as dwords (c01, c45, c23, c67),
// so one 16-byte read of a piece is the operand of a block pair.
__device__ __forceinline__ uint4 interleave_blocks(uint4 v) { return make_uint4(v.x, v.z, v.y, v.w); }

// The first n (< 16 / ES) elements of a 16-byte piece, zeros after them.
template <int ES>
__device__ __forceinline__ uint4 cut_piece(uint4 v, int n) {
  const int keep = n * ES;  // bytes
  const auto dw = [&](uint32_t x, int j) {
    const int kb = keep - 4 * j;
    return kb >= 4 ? x : (kb <= 0 ? 0u : x & ((1u << (8 * kb)) - 1u));
  };
  return make_uint4(dw(v.x, 0), dw(v.y, 1), dw(v.z, 2), dw(v.w, 3));
}

// One 16-byte halo piece whose channels are not all present or not 16-byte
// aligned: its first n_el (< 16 / ES) elements, zeros after them.  pairs
// (16-bit elements, even pitch and offset: the piece starts on a 4-byte
// boundary) reads two elements per 4-byte load; a last odd element's load
// also covers the element after it, which still lies inside the voxel's row
// (an even pitch leaves room for it) and is masked off.  Otherwise one load
// per element.
template <int ES>
__device__ __forceinline__ uint4 load_ragged(const uint8_t *src, int n_el, bool pairs) {
  constexpr int EPP = 16 / ES;
  uint32_t w[4] = {0u, 0u, 0u, 0u};
  if (ES == 2 && pairs) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (2 * q < n_el) {
        const uint32_t d = reinterpret_cast<const uint32_t *>(src)[q];
        w[q] = 2 * q + 1 < n_el ? d : (d & 0xffffu);
      }
    }
  } else {
#pragma unroll
    for (int e = 0; e < EPP; ++e) {
      if (e < n_el) {
        uint32_t bits;
        if constexpr (ES == 4) bits = reinterpret_cast<const uint32_t *>(src)[e];
        else bits = reinterpret_cast<const uint16_t *>(src)[e];
        w[(e * ES) >> 2] |= bits << (((e * ES) & 3) * 8);
      }
    }
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

template <int ES, bool ILV = false>
__device__ __forceinline__ void stage_halo(uint8_t *lds, const ConvArgs &a, const Brick &b,
                                           int c0) {
  constexpr int EPP = 16 / ES;                 // elements per 16-byte piece
  const int ppr = a.cc / EPP;                  // pieces per halo row
  const int total = a.ht * a.hh * a.hw * ppr;
  // vec: every piece that starts inside the layer's channels lies inside
  // its 16-byte aligned row (a ragged channel count's last piece is cut).
  const bool vec = (a.x_pitch % EPP) == 0 && (a.x_off % EPP) == 0;
  const bool pairs = ES == 2 && (a.x_pitch % 2) == 0 && (a.x_off % 2) == 0;
  const uint8_t *xb = static_cast<const uint8_t *>(a.x);
  for (int idx = threadIdx.x; idx < total; idx += blockDim.x) {
    const DivMod p = divmod(idx, ppr), x = divmod(p.q, a.hw), y = divmod(x.q, a.hh);
    const int hv = p.q, piece = p.r;
    const int xw = x.r, xh = y.r, xt = y.q;
    const int zt = b.zt0 + xt, zh = b.zh0 + xh, zw = b.zw0 + xw;
    const int c = c0 + piece * EPP;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (zt >= 0 && zt < a.t && zh >= 0 && zh < a.h && zw >= 0 && zw < a.w && c < a.c_in) {
      const long vox = ((static_cast<long>(b.nb) * a.t + zt) * a.h + zh) * a.w + zw;
      const uint8_t *src = xb + (vox * a.x_pitch + a.x_off + c) * ES;
      if (vec) {
        v = *reinterpret_cast<const uint4 *>(src);
        if (a.c_in - c < EPP) v = cut_piece<ES>(v, a.c_in - c);
      } else {
        v = load_ragged<ES>(src, min(EPP, a.c_in - c), pairs);
      }
    }
    if constexpr (ILV) v = interleave_blocks(v);
    *reinterpret_cast<uint4 *>(lds + hv * a.row + piece * 16) = v;  // rows are 16-byte multiples
  }
}

// Chunk stager with register prefetch.  Thread t owns the 16-byte halo
// pieces t + k*blockDim (k < MAXI).  init() resolves their input voxels once
// per workgroup; issue() starts the global loads of one channel chunk into
// registers (all of them back to back, so one memory latency per chunk);
// commit() writes them to LDS.  The kernels issue chunk c+1 before computing
// chunk c, so the loads overlap the MFMA work.  `ok` is false when the halo
// needs more than MAXI pieces per thread; the kernels then use stage_halo.
// FAST (c_in, the input pitch and the input offset multiples of the piece):
// every piece is one 16-byte load from
// a clamped, always valid address, and pieces that are padding are zeroed
// at commit, so the loads issue back to back without branches.
template <int ES, int MAXI, bool FAST = false, bool ILV = false>
struct Stager {
  static constexpr int EPP = 16 / ES;
  int vox[MAXI];   // flat input voxel; -1 padding (zeros); -2 no piece
  uint4 d[MAXI];
  int total, shift, ppr;
  unsigned live;   // FAST: bit k set when piece k holds input data
  bool ok;

  __device__ __forceinline__ void init(const ConvArgs &a, const Brick &b) {
    ppr = a.cc / EPP;  // a power of two
    shift = __builtin_ctz(static_cast<unsigned>(ppr));
    total = a.ht * a.hh * a.hw * ppr;
    ok = total <= MAXI * static_cast<int>(blockDim.x);
    // Halo row of piece k: (threadIdx.x + k * blockDim.x) >> shift, walked
    // with carries from one divmod pair (blockDim is a multiple of ppr).
    const DivMod x = divmod(static_cast<int>(threadIdx.x) >> shift, a.hw), y = divmod(x.q, a.hh);
    int xw = x.r, xh = y.r, xt = y.q;
    const int rstep = static_cast<int>(blockDim.x) >> shift;
    const DivMod sx = divmod(rstep, a.hw), sy = divmod(sx.q, a.hh);
#pragma unroll
    for (int k = 0; k < MAXI; ++k) {
      const int idx = threadIdx.x + k * blockDim.x;
      const int zt = b.zt0 + xt, zh = b.zh0 + xh, zw = b.zw0 + xw;
      const bool in = (static_cast<unsigned>(zt) < static_cast<unsigned>(a.t)) &
                      (static_cast<unsigned>(zh) < static_cast<unsigned>(a.h)) &
                      (static_cast<unsigned>(zw) < static_cast<unsigned>(a.w));
      vox[k] = idx < total ? (in ? ((b.nb * a.t + zt) * a.h + zh) * a.w + zw : -1) : -2;
      xw += sx.r;
      const int cw = xw >= a.hw ? 1 : 0;
      xw -= cw * a.hw;
      xh += sy.r + cw;
      const int chh = xh >= a.hh ? 1 : 0;
      xh -= chh * a.hh;
      xt += sy.q + chh;
    }
  }

  __device__ __forceinline__ void issue(const ConvArgs &a, int c0) {
    const uint8_t *xb = static_cast<const uint8_t *>(a.x);
    if constexpr (FAST) {
      unsigned bits = 0;
#pragma unroll
      for (int k = 0; k < MAXI; ++k) {
        // Rounds k with no piece in the whole workgroup issue no load (a
        // uniform branch: the halo size is the same for every thread).
        if (k * static_cast<int>(blockDim.x) >= total) break;
        const int idx = threadIdx.x + k * blockDim.x;
        const int c = c0 + (idx & (ppr - 1)) * EPP;
        const bool in = vox[k] >= 0 && c < a.c_in;
        const long el =
            static_cast<long>(max(vox[k], 0)) * a.x_pitch + a.x_off + min(c, a.c_in - EPP);
        d[k] = *reinterpret_cast<const uint4 *>(xb + el * ES);
        bits |= (in ? 1u : 0u) << k;
      }
      live = bits;
      return;
    }
    const bool vec = (a.x_pitch % EPP) == 0 && (a.x_off % EPP) == 0;  // as in stage_halo
    const bool pairs = ES == 2 && (a.x_pitch % 2) == 0 && (a.x_off % 2) == 0;
#pragma unroll
    for (int k = 0; k < MAXI; ++k) {
      const int idx = threadIdx.x + k * blockDim.x;
      const int c = c0 + (idx & (ppr - 1)) * EPP;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (vox[k] >= 0 && c < a.c_in) {
        const uint8_t *src = xb + (static_cast<long>(vox[k]) * a.x_pitch + a.x_off + c) * ES;
        if (vec) {
          v = *reinterpret_cast<const uint4 *>(src);
          if (a.c_in - c < EPP) v = cut_piece<ES>(v, a.c_in - c);
        } else {
          v = load_ragged<ES>(src, min(EPP, a.c_in - c), pairs);
        }
      }
      d[k] = v;
    }
  }

  __device__ __forceinline__ void commit(uint8_t *lds, const ConvArgs &a) const {
#pragma unroll
    for (int k = 0; k < MAXI; ++k) {
      const int idx = threadIdx.x + k * blockDim.x;
      if (vox[k] != -2) {
        uint4 v = d[k];
        if constexpr (FAST) {
          if (!((live >> k) & 1u)) v = make_uint4(0, 0, 0, 0);
        }
        if constexpr (ILV) v = interleave_blocks(v);
        *reinterpret_cast<uint4 *>(lds + (idx >> shift) * a.row + (idx & (ppr - 1)) * 16) = v;
      }
    }
  }
};

// ---------------------------------------------------------------------------
// Epilogue: y = act(acc + bias (+ residual)), four consecutive filters of one
// voxel per call.
// ---------------------------------------------------------------------------

template <typename T>
__device__ __forceinline__ float to_f32(T v) { return static_cast<float>(v); }

// Channel chunks handled by this workgroup's split (the host keeps nchunks
// below 4096, so the products stay in the 24-bit division's range).
__device__ __forceinline__ void split_range(const ConvArgs &a, int split, int &ch0, int &ch1) {
  ch0 = uniform(divmod(split * a.nchunks, a.splits).q);
  ch1 = uniform(divmod((split + 1) * a.nchunks, a.splits).q);
}

// ---------------------------------------------------------------------------
// Tile epilogue.  After the K loop every wave writes its fp32 accumulators
// into an LDS tile [voxel slot][filter of the workgroup]; the workgroup then
// stores it cooperatively, four consecutive filters per thread and item, so
// each 64-lane store covers whole output rows (channels-last).  On the way it
// adds bias and residual, applies ReLU, max-pools windows of qt x qh x qw
// voxels (bricks hold whole windows), rounds to the output dtype -- or, for a
// split of the channel range, stores the raw fp32 partial sums.
// ---------------------------------------------------------------------------

// act(acc + bias (+ residual)) for filters m0..m0+3 of unpooled voxel vox.
// Bias of filters m0..m0+3 (zero where absent).  Loaded once per thread and
// output column, outside the voxel loops.
// Completes, at this point, every load that writes v: an empty asm statement
// that reads a register makes the wait-count insertion wait for it here.
template <typename V>
__device__ __forceinline__ void settle(const V &v) {
  if constexpr (sizeof(V) == 16) {
    asm volatile("" ::"v"(__builtin_bit_cast(u32x4, v)));
  } else {
    static_assert(sizeof(V) == 8, "settle: 8 or 16 bytes");
    asm volatile("" ::"v"(__builtin_bit_cast(unsigned long long, v)));
  }
}

__device__ __forceinline__ float4 load_bias4(const ConvArgs &a, int m0) {
  float r[4] = {0.f, 0.f, 0.f, 0.f};
  if (a.bias && m0 < a.c_out) {
    if ((a.c_out & 3) == 0) {
      const float4 bb = *reinterpret_cast<const float4 *>(a.bias + m0);
      r[0] = bb.x; r[1] = bb.y; r[2] = bb.z; r[3] = bb.w;
    } else {
      for (int q = 0; q < 4; ++q)
        if (m0 + q < a.c_out) r[q] = a.bias[m0 + q];
    }
  }
  return make_float4(r[0], r[1], r[2], r[3]);
}

// RES = false compiles the residual path out (the caller knows a.res is NULL).
template <typename T, bool RES = true>
__device__ __forceinline__ float4 activate4(const ConvArgs &a, long vox, int m0, float4 v,
                                            float4 bb) {
  float r[4] = {v.x + bb.x, v.y + bb.y, v.z + bb.z, v.w + bb.w};
  const bool full = (a.c_out & 3) == 0;
  if (RES && a.res) {
    const T *res = static_cast<const T *>(a.res) + vox * a.c_out + m0;
    if (full && sizeof(T) == 4) {
      const float4 rr = *reinterpret_cast<const float4 *>(res);
      r[0] += rr.x; r[1] += rr.y; r[2] += rr.z; r[3] += rr.w;
    } else if (full) {
      union { uint2 u; T e[4]; } rr;
      rr.u = *reinterpret_cast<const uint2 *>(res);
      for (int q = 0; q < 4; ++q) r[q] += to_f32(rr.e[q]);
    } else {
      for (int q = 0; q < 4; ++q)
        if (m0 + q < a.c_out) r[q] += to_f32(res[q]);
    }
  }
  if (a.relu)
    for (int q = 0; q < 4; ++q) r[q] = r[q] > 0.f ? r[q] : 0.f;
  return make_float4(r[0], r[1], r[2], r[3]);
}

// Round and store filters m0..m0+3 of output voxel vox (of y's own extent).
template <typename T>
__device__ __forceinline__ void put4(const ConvArgs &a, long vox, int m0, float4 v) {
  T *y = static_cast<T *>(a.y) + vox * a.y_pitch + a.y_off + m0;
  const float r[4] = {v.x, v.y, v.z, v.w};
  if ((a.c_out & 3) == 0) {  // y_pitch and y_off are multiples of 4 as well
    if constexpr (sizeof(T) == 4) {
      *reinterpret_cast<float4 *>(y) = v;
    } else {
      union { uint2 u; T e[4]; } o;
      for (int q = 0; q < 4; ++q) o.e[q] = static_cast<T>(r[q]);
      *reinterpret_cast<uint2 *>(y) = o.u;
    }
  } else {
    for (int q = 0; q < 4 && m0 + q < a.c_out; ++q) y[q] = static_cast<T>(r[q]);
  }
}

__device__ __forceinline__ float4 max4(float4 x, float4 y) {
  return make_float4(x.x > y.x ? x.x : y.x, x.y > y.y ? x.y : y.y, x.z > y.z ? x.z : y.z,
                     x.w > y.w ? x.w : y.w);
}

__device__ __forceinline__ float4 add4(float4 x, float4 y) {
  return make_float4(x.x + y.x, x.y + y.y, x.z + y.z, x.w + y.w);
}

// v of lane l ^ 1: a quad permutation (1, 0, 3, 2) on the DPP path, without
// the LDS round trip of a general shuffle.  Lanes l and l ^ 1 must be both
// active.
__device__ __forceinline__ float swap_pair(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
}

__device__ __forceinline__ float4 swap_pairs4(float4 v) {
  return make_float4(swap_pair(v.x), swap_pair(v.y), swap_pair(v.z), swap_pair(v.w));
}

__device__ __forceinline__ float4 shfl_xor4(float4 v, int m) {
  return make_float4(__shfl_xor(v.x, m), __shfl_xor(v.y, m), __shfl_xor(v.z, m),
                     __shfl_xor(v.w, m));
}


// r[k] <- r[(k + by) % R] for a wave-uniform 0 <= by < R.
// Every lane of a quad takes lane P of the quad's value (DPP quad_perm).
template <int P>
__device__ __forceinline__ uint2 quad_bcast(uint2 v) {
  constexpr int ctrl = P | (P << 2) | (P << 4) | (P << 6);
  return make_uint2(
      static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v.x), ctrl, 0xF, 0xF, false)),
      static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v.y), ctrl, 0xF, 0xF, false)));
}

template <int R, typename X>
__device__ __forceinline__ void rotate_ring(X (&r)[R], int by) {
  static_for<R - 1>([&](auto kc) {
    constexpr int K = decltype(kc)::value + 1;
    if (by == K) {
      X t[R];
      static_for<R>([&](auto ic) { t[ic] = r[(decltype(ic)::value + K) % R]; });
      static_for<R>([&](auto ic) { r[ic] = t[ic]; });
    }
  });
}

// Walks voxel slots (t, h, w) of a bt x bh x bw box in steps of `step`
// slots with carries instead of divisions (step is at most 64).
struct BoxIter {
  int t, h, w;
  __device__ __forceinline__ void init(int slot, int bh, int bw) {
    const DivMod x = divmod(slot, bh * bw), y = divmod(x.r, bw);
    t = x.q;
    h = y.q;
    w = y.r;
  }
  __device__ __forceinline__ void advance(int step, int bh, int bw) {
    w += step;
    while (w >= bw) { w -= bw; ++h; }
    while (h >= bh) { h -= bh; ++t; }
  }
};

// Split-K partial of four consecutive filters of one voxel slot, stored
// straight from the accumulator registers (the reduction pass applies the
// epilogue, so no LDS tile is needed).
__device__ __forceinline__ void put_partial(const ConvArgs &a, const Slot &sl, int m0, int split,
                                            const f32x4 &v) {
  if (!sl.valid || m0 >= a.c_out) return;
  *reinterpret_cast<f32x4 *>(a.ws + (static_cast<long>(split) * a.total_vox + sl.out) * a.c_out4 + m0) = v;
}

// First filter (layer order) of 4-filter block slot `slot` of the wave
// tiles (slots 4*mfw*wt ... belong to wave tile wt): a union layout may have
// reordered the blocks so that tile-mates keep similar items.  Slots past
// the last wave tile (a workgroup's idle waves) stay past c_out.
__device__ __forceinline__ int block_filter0(const ConvArgs &a, int slot) {
  return 4 * (a.gmap && slot < a.gmap_slots ? static_cast<int>(a.gmap[slot]) : slot);
}

template <typename T>
__device__ __forceinline__ void tile_store(const ConvArgs &a, const Brick &b, const uint8_t *lds,
                                           int m_wg0) {
  // Thread t owns the 4-filter group t % cg of every voxel slot
  // t / cg + k * (blockDim / cg); cg divides the block size (16, 32 or 64).
  const int cg = a.c_wg >> 2;
  const int step = blockDim.x / cg;
  const int c4 = threadIdx.x % cg;
  const int m0 = block_filter0(a, (m_wg0 >> 2) + c4);
  const bool live = m0 < a.c_out;
  const float4 bb = load_bias4(a, m0);
  const uint8_t *col = lds + c4 * 16;
  const int pbt = a.bt / a.qt, pbh = a.bh / a.qh, pbw = a.bw / a.qw;
  const int npslots = pbt * pbh * pbw;
  BoxIter it;
  int ps = threadIdx.x / cg;
  it.init(ps, pbh, pbw);
  for (; ps < npslots; ps += step, it.advance(step, pbh, pbw)) {
    const int gt = b.ot0 / a.qt + it.t, gh = b.oh0 / a.qh + it.h, gw = b.ow0 / a.qw + it.w;
    if (!live || gt >= a.pto || gh >= a.pho || gw >= a.pwo) continue;
    float4 best = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int dt = 0; dt < a.qt; ++dt)
      for (int dh = 0; dh < a.qh; ++dh)
        for (int dw = 0; dw < a.qw; ++dw) {
          const int tt = it.t * a.qt + dt, hh = it.h * a.qh + dh, ww = it.w * a.qw + dw;
          const int slot = (tt * a.bh + hh) * a.bw + ww;
          const long vox = ((static_cast<long>(b.nb) * a.to + b.ot0 + tt) * a.ho + b.oh0 + hh) * a.wo + b.ow0 + ww;
          const float4 acc = *reinterpret_cast<const float4 *>(col + slot * a.tile_row);
          const float4 v = activate4<T>(a, vox, m0, acc, bb);
          best = (dt | dh | dw) ? max4(best, v) : v;
        }
    const long pvox = ((static_cast<long>(b.nb) * a.pto + gt) * a.pho + gh) * a.pwo + gw;
    put4<T>(a, pvox, m0, best);
  }
}

// ---------------------------------------------------------------------------
// 16-bit item kernel: v_mfma_f32_16x16x32_{bf16,f16}.
//
// A K-step is 8 items = 32 reduction slots.  Operand lane layouts (measured
// on gfx950): A[m][k] in lane m + 16*(k/8), element k%8; B[k][n] in lane
// n + 16*(k/8), element k%8; D[m][n] in lane n + 16*(m/4), element m%4.  So
// lane group g = lane/16 reads items 2g and 2g+1 (4 channels each, 8 bytes)
// for its voxel n, and the A stream is stored in exactly that lane order.
//
// The waves of a workgroup share one brick; wave w computes wave tile
// tg*wpw + w: 16*MFW filters x 16*NF voxel slots.  The split index selects
// a range of channel chunks (split-K) when the layer alone cannot fill the
// GPU.  Dense layers give every wave tile the
// full item list (and MFW > 1 shares each B fragment across filter rows);
// KGS layers give each 16-filter tile either the union of the items its four
// kernel groups keep, with the pruned entries of that union stored as zero
// weights, or (PAIR) the pair mapping below.
//
// PAIR: v_smfmac_f32_16x16x64_{bf16,f16}, 2:4 structured-sparse A.  A K-step
// is 8 pairs of items (64 reduction slots); the planner pairs two items only
// when no kernel group of the tile keeps both, so in every quad of four
// consecutive reduction slots a filter row has at most two nonzero weights,
// and a step multiplies up to 16 items in the time of one dense 16x16x32
// MFMA.  Reduction slots of pair j (items X, Y): quad 2j = (X.c0, X.c1, Y.c0,
// Y.c1), quad 2j+1 = (X.c2, X.c3, Y.c2, Y.c3).  Lane layouts (measured on
// gfx950): A (compressed, 8 values) lane m + 16*ga, element e -> quad
// 4*ga + e/2, so lane group ga holds pairs 2ga and 2ga+1 of its filter row;
// B lane n + 16*gb, element e -> slot 8*gb + e (e < 8) or 32 + 8*gb + e - 8,
// so lane group gb reads pairs gb and gb+4 (four 8-byte LDS reads); the
// 2-bit index of element e sits at bits 2e of the index register (ABID 0).
// Weights stream compact: one 32-byte 4x4 block per kept (pair, group).  Per
// step and (lane group, kernel group) the planner stores the byte offsets of
// the blocks of the lane group's two pairs and their index register; a group
// that keeps neither item of a pair gets an offset beyond the buffer's
// extent, which loads zeros without touching memory, so pruned weights never
// leave HBM.
// ---------------------------------------------------------------------------

// FAST: c_in is a multiple of 8 (branch-free halo staging).
// MAP: 0 = dense / KGS union, 1 = pairs of any two items, 2 = block pairs.
// The pair mappings, the 64-slot tiles and the two-row 128-slot tiles ask
// for two waves per SIMD: left to itself the compiler spends registers down
// to one wave (the pairs' index registers ride with A; the union's unrolled
// passes lengthen live ranges; two rows of eight fragments spill a few
// registers to fit), and a lone wave cannot hide its LDS reads behind the
// other's MFMAs.
template <typename T, int MFW, int NF, bool FAST, int MAP = 0>
__global__ __launch_bounds__(256, (MAP != 0 || NF == 4 || MFW == 2) ? 2 : 1) void items16_kernel(ConvArgs a) {
  constexpr bool PAIR = MAP != 0;
  constexpr bool BPAIR = MAP == 2;
  // Pairs of any two items on 16-filter tiles stream compact weights; wide
  // pair tiles and block pairs stream weights and index registers in lane
  // order.
  constexpr bool COMPACT = MAP == 1 && MFW == 1;
  using V8 = std::conditional_t<std::is_same_v<T, __bf16>, bf16x8, f16x8>;
  using V16 = std::conditional_t<std::is_same_v<T, __bf16>, bf16x16, f16x16>;
  using BV = std::conditional_t<PAIR, V16, V8>;     // B fragment of one step
  // LDS offsets of a lane group's reads: 2 items (union), the X and Y items
  // of 2 pairs (pairs), 2 block pairs (block pairs)
  using OFF = std::conditional_t<MAP == 1, uint4, uint2>;
  // Software pipeline of a wave (step t = one K-step of 8 items):
  //   item offsets four or more steps ahead and the A operand for step t+2
  //   are in flight from global memory, and the B fragments of step t+1 are
  //   read from LDS, while the MFMAs of step t run.  Rings: A 2, B 2;
  //   offsets 4 (pair mappings) or two blocks of four steps (union / dense).
  extern __shared__ __align__(16) uint8_t lds[];
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  const Wg wg = decode_wg(a);
  const int wt = uniform(wg.tg * a.wpw + (static_cast<int>(threadIdx.x) >> 6));
  const bool active = wt < a.wave_tiles;
  const Brick b = decode_brick(a, wg.brick);

  int vb[NF];
  {
    SlotWalk sw;
    sw.init(a, lane & 15, 16);
#pragma unroll
    for (int j = 0; j < NF; ++j) {
      vb[j] = slot_lds(a, b, sw.t, sw.h, sw.w);
      sw.next(a);
    }
  }

  // First filter (layer order) of this lane's 4-filter block in each row.
  int mf0[MFW];
#pragma unroll
  for (int i = 0; i < MFW; ++i) mf0[i] = block_filter0(a, wt * 4 * MFW + 4 * i + g);

  f32x4 acc[MFW][NF];
  #pragma unroll
  for (int i = 0; i < MFW; ++i)
    #pragma unroll
    for (int j = 0; j < NF; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const uint32_t *sp = a.step_ptr + static_cast<long>(active ? wt : 0) * (a.nchunks + 1);
  const uint32_t step0 = uniform(sp[0]);
  const uint32_t row0 = uniform(a.item_ptr[active ? wt : 0]);
  const V8 *A = static_cast<const V8 *>(a.a) + lane;
  // Union / dense: 8 item offsets per step, lane group g reads 2 of them;
  // PAIR: 16 per step, lane group g reads the items of pairs g and g + 4.
  const OFF *IT = reinterpret_cast<const OFF *>(a.items) + g;

  OFF roff[4];
  V8 ra[2][MFW];
  BV rb[2][NF];
  // PAIR: each A slot carries its 2-bit index registers; the compact stream's
  // step descriptors ride with the offsets.
  uint4 rdesc[COMPACT ? 4 : 1];
  uint32_t ridx[2][MFW] = {};
  const uint32_t *IDX = a.keep + lane;  // PAIR, MFW > 1: [step][i][lane]
  const uint32_t row8 = (lane & 3) * 8u;           // this lane's filter row within a block
  const __amdgpu_buffer_rsrc_t ares =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(a.a), 0, static_cast<int>(a.a_bytes), 0x00020000);
  // PAIR: this lane's descriptor {block offset of pair 2g, of pair 2g + 1,
  // index register, 0} of step s is entry 16 s + 4 g + (kernel group).
  const uint4 *KD = reinterpret_cast<const uint4 *>(a.keep) + 4 * g + ((lane & 15) >> 2);
  auto fetch_off = [&](int slot, uint32_t s) {
    roff[slot] = IT[(static_cast<long>(row0) + (s - step0)) * 4];
    if constexpr (COMPACT) rdesc[slot] = KD[static_cast<long>(s) * 16];
  };
  // dslot: the offsets-ring slot that holds step s's descriptor (PAIR).
  auto fetch_a = [&](int slot, uint32_t s, int dslot) {
    if constexpr (COMPACT) {
      // This lane's filter row of the two blocks (offsets >= 2^31 read zeros).
      const uint4 d = rdesc[dslot];
      const uint2 lo = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(ares, static_cast<int>(d.x + row8), 0, 0));
      const uint2 hi = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(ares, static_cast<int>(d.y + row8), 0, 0));
      ra[slot][0] = __builtin_bit_cast(V8, make_uint4(lo.x, lo.y, hi.x, hi.y));
      ridx[slot][0] = d.z;
    } else {
      (void)dslot;
      #pragma unroll
      for (int i = 0; i < MFW; ++i) {
        ra[slot][i] = A[(static_cast<long>(s) * MFW + i) * 64];
        if constexpr (PAIR) ridx[slot][i] = IDX[(static_cast<long>(s) * MFW + i) * 64];
      }
    }
  };
  auto load_b = [&](int slot, OFF off) {
    #pragma unroll
    for (int j = 0; j < NF; ++j) {
      if constexpr (BPAIR) {
        // One 16-byte read per block pair: the staged interleave makes it
        // (X.c01, Y.c01, X.c23, Y.c23), the operand order.
        const uint4 p0 = *reinterpret_cast<const uint4 *>(lds + vb[j] + off.x);
        const uint4 p1 = *reinterpret_cast<const uint4 *>(lds + vb[j] + off.y);
        rb[slot][j] = __builtin_bit_cast(V16, u32x8{p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w});
      } else if constexpr (PAIR) {
        // Two 8-byte reads per pair; operand order is (X.c01, Y.c01, X.c23,
        // Y.c23).  Wide tiles keep the reads in load order (X.c01, X.c23,
        // Y.c01, Y.c23), landing in place, and swap them in the MFMA stage a
        // step later (swapping here waits for the reads every step; measured
        // 808 -> 761 us on batch-32 conv3b); 16-filter tiles swap here (the
        // deferred swap's extra registers cost them: conv2 54 -> 82 us).
        // LDS time follows the number of read instructions more than their
        // width: four 4-byte reads per pair that would land in operand order
        // measured about twice as slow.
        const uint2 x0 = *reinterpret_cast<const uint2 *>(lds + vb[j] + off.x);
        const uint2 y0 = *reinterpret_cast<const uint2 *>(lds + vb[j] + off.y);
        const uint2 x1 = *reinterpret_cast<const uint2 *>(lds + vb[j] + off.z);
        const uint2 y1 = *reinterpret_cast<const uint2 *>(lds + vb[j] + off.w);
        if constexpr (MFW > 1)
          rb[slot][j] = __builtin_bit_cast(V16, u32x8{x0.x, x0.y, y0.x, y0.y, x1.x, x1.y, y1.x, y1.y});
        else
          rb[slot][j] = __builtin_bit_cast(V16, u32x8{x0.x, y0.x, x0.y, y0.y, x1.x, y1.x, x1.y, y1.y});
      } else {
        const uint2 lo = *reinterpret_cast<const uint2 *>(lds + vb[j] + off.x);
        const uint2 hi = *reinterpret_cast<const uint2 *>(lds + vb[j] + off.y);
        rb[slot][j] = __builtin_bit_cast(V8, make_uint4(lo.x, lo.y, hi.x, hi.y));
      }
    }
  };
  auto mma = [&](int slot) {
    #pragma unroll
    for (int j = 0; j < NF; ++j) {
      BV bj = rb[slot][j];
      if constexpr (MAP == 1 && MFW > 1) {
        // load order (X.c01, X.c23, Y.c01, Y.c23) -> quads (X.c01, Y.c01), (X.c23, Y.c23)
        u32x8 r = __builtin_bit_cast(u32x8, bj);
        bj = __builtin_bit_cast(V16, u32x8{r[0], r[2], r[1], r[3], r[4], r[6], r[5], r[7]});
      }
      #pragma unroll
      for (int i = 0; i < MFW; ++i) {
        if constexpr (PAIR) {
          if constexpr (std::is_same_v<T, __bf16>)
            acc[i][j] = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(ra[slot][i], bj, acc[i][j],
                                                                   static_cast<int>(ridx[slot][i]), 0, 0);
          else
            acc[i][j] = __builtin_amdgcn_smfmac_f32_16x16x64_f16(ra[slot][i], bj, acc[i][j],
                                                                  static_cast<int>(ridx[slot][i]), 0, 0);
        } else if constexpr (std::is_same_v<T, __bf16>) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ra[slot][i], bj, acc[i][j], 0, 0, 0);
        } else {
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ra[slot][i], bj, acc[i][j], 0, 0, 0);
        }
      }
    }
  };

  int ch0, ch1;
  split_range(a, wg.split, ch0, ch1);
  // The wave's steps over all chunks of its split form one stream
  // [S0, S1) (indices clamped to the last step: a harmless re-read, so the
  // loop bodies stay straight-line and the wait counters exact).  The pair
  // mappings prefetch offsets and A along it straight across chunk
  // boundaries; union / dense reload the next chunk's first offsets and A
  // slots at each chunk's end, so that their step tail can run branch-free.
  // Only the B fragments wait for a new chunk to reach LDS.
  const uint32_t S0 = uniform(sp[ch0]), S1 = uniform(sp[ch1]);
  const bool work = active && S1 > S0;
  const uint32_t LAST = work ? S1 - 1 : S0;
  Stager<2, 8, FAST, BPAIR> st;
  st.init(a, b);
  if (st.ok && ch0 < ch1) st.issue(a, ch0 * a.cc);
  // Union / dense: the item offsets travel in blocks of four steps.  Lane
  // (n, g) of a block holds the two offsets of step base + (n & 3) for its
  // lane group g, and a quad broadcast (DPP) hands step base + d to all four
  // lanes of a quad, so one load serves four steps.  ob[0] and ob[1] hold
  // the blocks at chunk-relative steps 0 and 4 of each group of eight.
  uint2 ob[2];
  const uint2 *ITB = reinterpret_cast<const uint2 *>(a.items) + g;
  auto fetch_blk = [&](int slot, uint32_t base) {
    const uint32_t sl = min(base + static_cast<uint32_t>(lane & 3), LAST);
    ob[slot] = ITB[(static_cast<long>(row0) + (sl - step0)) * 4];
  };
  if (work) {
    if constexpr (MAP == 0) {
      fetch_blk(0, S0);
      fetch_blk(1, S0 + 4);
    } else {
#pragma unroll
      for (int d = 0; d < 4; ++d) fetch_off(d, min(S0 + d, LAST));
    }
#pragma unroll
    for (int d = 0; d < 2; ++d) fetch_a(d, min(S0 + d, LAST), d);
  }
  for (int ch = ch0; ch < ch1; ++ch) {
    __syncthreads();  // every wave is done with the previous chunk
    if (st.ok) st.commit(lds, a);
    else stage_halo<2, BPAIR>(lds, a, b, ch * a.cc);
    __syncthreads();
    if (st.ok && ch + 1 < ch1) st.issue(a, (ch + 1) * a.cc);  // overlaps this chunk's MFMAs
    if (!work) continue;
    const uint32_t s_beg = uniform(sp[ch]), s_end = uniform(sp[ch + 1]);
    if (s_beg == s_end) continue;
    if constexpr (MAP == 0) {
      // Local step i: A slot i&1, B slot i&1, offsets from block (i >> 2) & 1
      // at quad position i & 3.  Eight steps per pass; block 0 is refilled
      // after its last use (step 3) with steps 8..11, block 1 after step 7
      // with steps 12..15.
      load_b(0, quad_bcast<0>(ob[0]));
      uint32_t s = s_beg;
      for (; s + 8 <= s_end; s += 8) {
        static_for<8>([&](auto dc) {
          constexpr int D = decltype(dc)::value;
          load_b((D + 1) & 1, quad_bcast<(D + 1) & 3>(ob[((D + 1) >> 2) & 1]));
          mma(D & 1);
          fetch_a(D & 1, min(s + D + 2, LAST), 0);
          if constexpr (D == 3) fetch_blk(0, s + 8);
          if constexpr (D == 7) fetch_blk(1, s + 12);
          __builtin_amdgcn_sched_barrier(0);
        });
      }
      // 0..7 steps remain: one pass of four when at least four do, then up
      // to three.  The last three issue every load whether or not its step
      // exists (addresses clamped; unused data is never read) and only their
      // MFMAs depend on the step count, so their waits stay exact.
      const uint32_t rem = s_end - s;
      if (rem >= 4) {
        static_for<4>([&](auto dc) {
          constexpr int D = decltype(dc)::value;
          load_b((D + 1) & 1, quad_bcast<(D + 1) & 3>(ob[(D + 1) >> 2]));
          mma(D & 1);
          fetch_a(D & 1, min(s + D + 2, LAST), 0);
          __builtin_amdgcn_sched_barrier(0);
        });
        s += 4;
      }
      const bool hi = rem >= 4;
      const uint2 b0 = ob[0], b1 = ob[1];
      const uint2 blk = make_uint2(hi ? b1.x : b0.x, hi ? b1.y : b0.y);
      const uint32_t r = rem & 3;
      static_for<3>([&](auto dc) {
        constexpr int D = decltype(dc)::value;
        if constexpr (D < 2) load_b((D + 1) & 1, quad_bcast<D + 1>(blk));
        if (D < r) mma(D & 1);
        if constexpr (D == 0) fetch_a(0, min(s + 2, LAST), 0);
        __builtin_amdgcn_sched_barrier(0);
      });
      // The next chunk starts at s_end: load its first A slots and offset
      // blocks now (they land during the chunk barrier).
      fetch_a(0, min(s_end, LAST), 0);
      fetch_a(1, min(s_end + 1, LAST), 0);
      fetch_blk(0, s_end);
      fetch_blk(1, s_end + 4);
      continue;
    }
    // Ring slots are relative to the chunk's first step: offsets slot i&3,
    // A slot i&1, B slot i&1 for local step i.
    load_b(0, roff[0]);
    uint32_t s = s_beg;
    for (; s + 4 <= s_end; s += 4) {
      static_for<4>([&](auto dc) {
        constexpr int D = decltype(dc)::value;
        load_b((D + 1) & 1, roff[(D + 1) & 3]);
        mma(D & 1);
        fetch_a(D & 1, min(s + D + 2, LAST), (D + 2) & 3);
        fetch_off(D, min(s + D + 4, LAST));
        // Keep the stages in place: without this fence the scheduler sinks
        // the prefetches next to their uses two steps later.
        __builtin_amdgcn_sched_barrier(0);
      });
    }
    const uint32_t rem = s_end - s;  // tail: 0..3 steps
    static_for<3>([&](auto dc) {
      constexpr int D = decltype(dc)::value;
      if (D < rem) {
        if (D + 1 < rem) load_b((D + 1) & 1, roff[(D + 1) & 3]);
        mma(D & 1);
        fetch_a(D & 1, min(s + D + 2, LAST), (D + 2) & 3);
        fetch_off(D, min(s + D + 4, LAST));
      }
    });
    // The rings now hold steps s_end.. at slots (n + k) & 3 and (n + k) & 1
    // (n = steps of this chunk): rotate them to slot 0 for the next chunk.
    const uint32_t n = s_end - s_beg;
    rotate_ring(roff, static_cast<int>(n & 3));
    if constexpr (COMPACT) rotate_ring(rdesc, static_cast<int>(n & 3));
    if (n & 1) {
#pragma unroll
      for (int i = 0; i < MFW; ++i) {
        const V8 t = ra[0][i];
        ra[0][i] = ra[1][i];
        ra[1][i] = t;
        const uint32_t ti = ridx[0][i];
        ridx[0][i] = ridx[1][i];
        ridx[1][i] = ti;
      }
    }
  }
  if (a.splits > 1) {
    if (active) {
      SlotWalk sw;
      sw.init(a, lane & 15, 16);
#pragma unroll
      for (int j = 0; j < NF; ++j) {
        const Slot sl = slot_at(a, b, sw.t, sw.h, sw.w);
        sw.next(a);
#pragma unroll
        for (int i = 0; i < MFW; ++i)
          put_partial(a, sl, mf0[i], wg.split, acc[i][j]);
      }
    }
    return;
  }
  if (NF == 4 && MFW <= 4 && a.qt * a.qh * a.qw == 1) {
    // No pooling: a lane's accumulator holds 4 consecutive filters of one
    // voxel slot, so the epilogue runs on registers and stores straight to
    // y (no LDS tile, no barriers).
    if (active) {
      float4 bb[MFW];
#pragma unroll
      for (int i = 0; i < MFW; ++i) bb[i] = load_bias4(a, mf0[i]);
      SlotWalk sw;
      sw.init(a, lane & 15, 16);
#pragma unroll
      for (int j = 0; j < NF; ++j) {
        const Slot sl = slot_at(a, b, sw.t, sw.h, sw.w);
        sw.next(a);
        if (!sl.valid) continue;
#pragma unroll
        for (int i = 0; i < MFW; ++i) {
          const int m0 = mf0[i];
          if (m0 >= a.c_out) continue;
          const float4 raw = make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
          put4<T>(a, sl.out, m0, activate4<T>(a, sl.out, m0, raw, bb[i]));
        }
      }
    }
    return;
  }
  if (a.qt == 2 && a.qh == 2 && a.qw == 2 && a.bt == NF / 2 && a.bh == 2 && a.bw == 16) {
    // 2x2x2 pooling on a (NF/2)x2x16 brick: fragment j is the w-row (t, h) =
    // (j / 2, j % 2) and lane n its voxel w, so a window is fragments 4p ..
    // 4p + 3 of lanes n and n ^ 1 (every voxel of an output window lies
    // inside the output; other lanes' values are never stored).
    if (active) {
      const int n = lane & 15;
#pragma unroll
      for (int i = 0; i < MFW; ++i) {
        const int m0 = mf0[i];
        if (m0 >= a.c_out) continue;
        const float4 bb = load_bias4(a, m0);
#pragma unroll
        for (int p = 0; p < NF / 4; ++p) {
          float4 best = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const int j = 4 * p + k;
            const int ot = b.ot0 + (j >> 1), oh = b.oh0 + (j & 1), ow = b.ow0 + n;
            const bool ok = ot < a.to && oh < a.ho && ow < a.wo;
            const long vox = ((static_cast<long>(b.nb) * a.to + ot) * a.ho + oh) * a.wo + ow;
            const float4 raw = make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
            const float4 v = ok ? activate4<T>(a, vox, m0, raw, bb) : raw;
            best = k ? max4(best, v) : v;
          }
          best = max4(best, swap_pairs4(best));  // lanes n, n ^ 1 share g: both active
          const int pt = (b.ot0 >> 1) + p, ph = b.oh0 >> 1, pw = (b.ow0 + n) >> 1;
          if ((n & 1) == 0 && pt < a.pto && ph < a.pho && pw < a.pwo)
            put4<T>(a, ((static_cast<long>(b.nb) * a.pto + pt) * a.pho + ph) * a.pwo + pw, m0, best);
        }
      }
    }
    return;
  }
  const int m_wg0 = wg.tg * a.wpw * 16 * MFW;
  __syncthreads();  // the halo is no longer needed: reuse LDS for the tile
  if (active) {
#pragma unroll
    for (int j = 0; j < NF; ++j)
#pragma unroll
      for (int i = 0; i < MFW; ++i) {
        const int col = wt * 16 * MFW - m_wg0 + 16 * i + 4 * g;
        *reinterpret_cast<f32x4 *>(lds + (16 * j + (lane & 15)) * a.tile_row + col * 4) = acc[i][j];
      }
  }
  __syncthreads();
  tile_store<T>(a, b, lds, m_wg0);
}

// ---------------------------------------------------------------------------
// Small-input-channel kernel (c_in <= 4, at most 4 K-steps: a first layer on
// RGB clips).  Here the per-workgroup fixed cost of the item kernel (halo
// staging latency, barriers, the LDS output tile) dwarfs the 4 K-steps, so
// each wave works alone: it keeps its whole weight tile (16*MFW filters x all
// steps) in registers, owns a double-buffered halo in LDS, and walks bricks
// of 1 x 2 x 32 output voxels (64 slots, 4 fragments) with the next brick's
// input loads in flight while it computes and stores the current one.  Max
// pooling with a 1x2x2 window is done in registers (the h pair is two
// fragments of the same lane, the w pair two adjacent lanes).
// Halo rows hold 4 channels (8 bytes); channels >= c_in stay zero.
// ---------------------------------------------------------------------------

constexpr int kSmallLines = 12;      // halo lines (t, h) per brick: kt * (sh + kh) <= 12

// RES: the layer adds a residual (a separate instantiation keeps the common
// epilogue short).  STEPS: K-steps held in registers (4: kernels up to 32
// taps; 8: up to 64, e.g. the 1x7x7 stem convs).  EPL: halo elements per
// lane and line (2: one dword load, lines up to 127 elements; 4: one 8-byte
// load, up to 253).
template <typename T, int MFW, bool RES, int STEPS, int EPL>
__global__ __launch_bounds__(256) void small_kernel(ConvArgs a) {
  using V8 = std::conditional_t<std::is_same_v<T, __bf16>, bf16x8, f16x8>;
  constexpr int NF = 4;
  extern __shared__ __align__(16) uint8_t lds[];
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  const int wave = static_cast<int>(threadIdx.x) >> 6;
  const int rows = a.ht * a.hh * a.hw;
  // + a sink for elements outside the line: a 2-byte slot per lane, so that
  // the writes that land there do not collide in one bank
  const int buf_bytes = ((rows * 8 + 15) & ~15) + 128;
  uint8_t *mine = lds + wave * 2 * buf_bytes;
  for (int i = lane; i < 2 * buf_bytes / 16; i += 64)
    reinterpret_cast<uint4 *>(mine)[i] = make_uint4(0, 0, 0, 0);

  // Work split: wave gw handles wave tile gw % wave_tiles and bricks
  // gw / wave_tiles + k * (waves / wave_tiles); the host makes the wave
  // count a multiple of wave_tiles.
  const int gw = static_cast<int>(blockIdx.x) * 4 + wave;
  const int nwaves = static_cast<int>(gridDim.x) * 4;
  const int wt = uniform(gw % a.wave_tiles);
  const int bstride = uniform(nwaves / a.wave_tiles);
  int brick = uniform(gw / a.wave_tiles);

  // Weights and item offsets of the whole K loop, in registers.
  const uint32_t *sp = a.step_ptr + static_cast<long>(wt) * (a.nchunks + 1);
  const uint32_t s0 = uniform(sp[0]);
  const int steps = uniform(static_cast<int>(sp[1] - s0));
  const uint32_t row0 = uniform(a.item_ptr[wt]);
  const V8 *A = static_cast<const V8 *>(a.a) + lane;
  const uint2 *IT = reinterpret_cast<const uint2 *>(a.items) + g;
  V8 ra[STEPS][MFW];
  uint2 off[STEPS];
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    const uint32_t st = s0 + static_cast<uint32_t>(s < steps ? s : 0);
#pragma unroll
    for (int i = 0; i < MFW; ++i) ra[s][i] = A[(static_cast<long>(st) * MFW + i) * 64];
    off[s] = IT[(static_cast<long>(row0) + (st - s0)) * 4];
  }

  // Bias of this lane's filters.
  float4 bb[MFW];
#pragma unroll
  for (int i = 0; i < MFW; ++i) bb[i] = load_bias4(a, wt * 16 * MFW + 16 * i + 4 * g);

  // Let these loads land before the brick loop: the wait counters are
  // in-order, so a register still pending at the loop head would make the
  // MFMAs and the epilogue wait for every staging load issued after it.
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
#pragma unroll
    for (int i = 0; i < MFW; ++i) settle(ra[s][i]);
    settle(off[s]);
  }
#pragma unroll
  for (int i = 0; i < MFW; ++i) settle(bb[i]);

  // LDS row of each fragment's voxel slot (slot 16j + n of the 1x2x32 brick).
  int vb[NF];
#pragma unroll
  for (int j = 0; j < NF; ++j) {
    const int hh = j >> 1, ww = 16 * (j & 1) + (lane & 15);
    vb[j] = (hh * a.sh * a.hw + ww * a.sw) * 8;
  }

  // Halo staging.  Line L = (xt, xh) of a brick holds hw voxels x c_in
  // channels, contiguous in the channels-last input from element
  // E0 = (((n t + xt) h + xh) w + zw0) c_in.  A lane loads the aligned word
  // of EPL elements (E0 / EPL) + lane, i.e. line elements
  // e = EPL lane + u - E0 % EPL, u < EPL, so one load per lane covers a line
  // of up to 64 EPL - EPL + 1 elements; w c_in % 4 == 0 (host) gives every
  // line of a brick the same shift (zw0 c_in) % EPL and makes the input a
  // whole number of 8-byte words.  The loads go through a buffer resource
  // whose extent is the input: words before or past it, and whole lines
  // outside the clip (given an out-of-range offset), read as zero without
  // touching memory.  Element u of a lane lands at LDS byte pend[u] of its
  // line (voxel e / c_in, 8-byte rows of 4 channels), with bit 0 set when the
  // voxel is a padding column (a zero is staged), or in the lane's sink slot
  // when e is outside the line (pend[u] < 0).
  using W = std::conditional_t<EPL == 4, uint2, uint32_t>;
  const int line_len = a.hw * a.c_in;
  const long xbytes = static_cast<long>(a.n) * a.t * a.h * a.w * a.c_in * 2;  // < 2^31 - 8 (host)
  // Raw buffer (stride 0): the range check compares each word's byte offset
  // with the extent; the last descriptor word selects the 32-bit data format
  // that untyped loads use on this architecture.
  const __amdgpu_buffer_rsrc_t xres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(a.x), 0, static_cast<int>(xbytes), 0x00020000);
  const int nlines = a.ht * a.hh;
  const int sink = buf_bytes - 128 + 2 * lane;
  W sv[kSmallLines];
  int pend[EPL];
  auto issue = [&](int br) {
    const Brick b = decode_brick(a, br);
#pragma unroll
    for (int L = 0; L < kSmallLines; ++L) {
      const DivMod lt = divmod(L, a.hh);
      const int zt = b.zt0 + lt.q, zh = b.zh0 + lt.r;
      const bool line_ok = L < nlines && zt >= 0 && zt < a.t && zh >= 0 && zh < a.h;
      const int e0 = uniform((((b.nb * a.t + zt) * a.h + zh) * a.w + b.zw0) * a.c_in);
      const int base = line_ok ? 2 * EPL * (e0 >> (EPL == 4 ? 2 : 1)) : static_cast<int>(0x80000000u);
      if constexpr (EPL == 4)
        sv[L] = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(xres, base + 8 * lane, 0, 0));
      else
        sv[L] = __builtin_amdgcn_raw_buffer_load_b32(xres, base + 4 * lane, 0, 0);
    }
    const int shift = (b.zw0 * a.c_in) & (EPL - 1);
#pragma unroll
    for (int u = 0; u < EPL; ++u) {
      const int e = EPL * lane + u - shift;
      const DivMod d = divmod(max(e, 0), a.c_in);
      const bool pad = static_cast<unsigned>(b.zw0 + d.q) >= static_cast<unsigned>(a.w);
      pend[u] = static_cast<unsigned>(e) < static_cast<unsigned>(line_len) ? d.q * 8 + d.r * 2 + (pad ? 1 : 0)
                                                                           : -2;
    }
  };

  auto commit = [&](uint8_t *buf) {
#pragma unroll
    for (int L = 0; L < kSmallLines; ++L) {
      uint32_t half[EPL];
      if constexpr (EPL == 4) {
        half[0] = sv[L].x & 0xffffu;
        half[1] = sv[L].x >> 16;
        half[2] = sv[L].y & 0xffffu;
        half[3] = sv[L].y >> 16;
      } else {
        half[0] = sv[L] & 0xffffu;
        half[1] = sv[L] >> 16;
      }
#pragma unroll
      for (int u = 0; u < EPL; ++u) {
        const int o = L < nlines && pend[u] >= 0 ? L * a.hw * 8 + (pend[u] & ~1) : sink;
        *reinterpret_cast<uint16_t *>(buf + o) = static_cast<uint16_t>((pend[u] & 1) ? 0u : half[u]);
      }
    }
  };
  auto wave_sync = [] {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };

  int cur = 0;
  if (brick < a.nbricks) {
    issue(brick);
    wave_sync();  // zero fill done before the first commit
    commit(mine);
  }
  for (; brick < a.nbricks; brick += bstride) {
    // The next brick's loads are in flight during this brick.  The commit
    // below runs on every path (after the last brick it rewrites the idle
    // buffer with stale values): a conditional commit would look to the
    // wait-count insertion like loads that may skip their wait, and it would
    // then wait for them at the next issue and in the epilogue.
    const int next = brick + bstride;
    if (next < a.nbricks) issue(next);
    wave_sync();
    const uint8_t *buf = mine + cur * buf_bytes;
    f32x4 acc[MFW][NF];
#pragma unroll
    for (int i = 0; i < MFW; ++i)
#pragma unroll
      for (int j = 0; j < NF; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      if (s < steps) {
#pragma unroll
        for (int j = 0; j < NF; ++j) {
          const uint2 lo = *reinterpret_cast<const uint2 *>(buf + vb[j] + off[s].x);
          const uint2 hi = *reinterpret_cast<const uint2 *>(buf + vb[j] + off[s].y);
          const V8 bv = __builtin_bit_cast(V8, make_uint4(lo.x, lo.y, hi.x, hi.y));
#pragma unroll
          for (int i = 0; i < MFW; ++i) {
            if constexpr (std::is_same_v<T, __bf16>)
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ra[s][i], bv, acc[i][j], 0, 0, 0);
            else
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ra[s][i], bv, acc[i][j], 0, 0, 0);
          }
        }
      }
    }
    // Epilogue: activation per voxel, optional 1x2x2 max, store.
    const Brick b = decode_brick(a, brick);
    const int n = lane & 15;
#pragma unroll
    for (int i = 0; i < MFW; ++i) {
      const int m0 = wt * 16 * MFW + 16 * i + 4 * g;
      if (m0 >= a.c_out) continue;
      float4 v[NF];
      bool ok[NF];
      auto voxel = [&](int j) {
        return ((static_cast<long>(b.nb) * a.to + b.ot0) * a.ho + b.oh0 + (j >> 1)) * a.wo +
               b.ow0 + 16 * (j & 1) + n;
      };
#pragma unroll
      for (int j = 0; j < NF; ++j) {
        const int oh = b.oh0 + (j >> 1), ow = b.ow0 + 16 * (j & 1) + n;
        ok[j] = b.ot0 < a.to && oh < a.ho && ow < a.wo;
        const float4 raw = make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
        v[j] = ok[j] ? activate4<T, RES>(a, voxel(j), m0, raw, bb[i]) : raw;
      }
      if (a.qh == 2) {  // window 1x2x2 (bricks hold whole windows)
#pragma unroll
        for (int jw = 0; jw < 2; ++jw) {
          float4 m = max4(v[jw], v[jw + 2]);
          m = max4(m, swap_pairs4(m));  // lanes n, n ^ 1 share g: both active
          const int ow = b.ow0 + 16 * jw + n;
          const int ph = b.oh0 >> 1, pw = ow >> 1;
          if ((n & 1) == 0 && b.ot0 < a.pto && ph < a.pho && pw < a.pwo)
            put4<T>(a, ((static_cast<long>(b.nb) * a.pto + b.ot0) * a.pho + ph) * a.pwo + pw, m0, m);
        }
      } else {
#pragma unroll
        for (int j = 0; j < NF; ++j)
          if (ok[j]) put4<T>(a, voxel(j), m0, v[j]);
      }
    }
    cur ^= 1;
    commit(mine + cur * buf_bytes);
  }
}

// ---------------------------------------------------------------------------
// f32 dense item kernel: v_mfma_f32_16x16x4_f32 (full fp32, no reduced
// precision).  A K-step is 4 items = 16 reduction slots issued as four
// MFMAs; in MFMA s lane group g supplies channel s of item g, so one
// 16-byte LDS read per lane feeds all four.
// ---------------------------------------------------------------------------

template <int MFW, int NF>
__global__ __launch_bounds__(256) void items_f32_kernel(ConvArgs a) {
  constexpr int DEPTH = 3;
  extern __shared__ __align__(16) uint8_t lds[];
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  const Wg wg = decode_wg(a);
  const int wt = uniform(wg.tg * a.wpw + (static_cast<int>(threadIdx.x) >> 6));
  const bool active = wt < a.wave_tiles;
  const Brick b = decode_brick(a, wg.brick);

  int vb[NF];
  {
    SlotWalk sw;
    sw.init(a, lane & 15, 16);
#pragma unroll
    for (int j = 0; j < NF; ++j) {
      vb[j] = slot_lds(a, b, sw.t, sw.h, sw.w);
      sw.next(a);
    }
  }

  f32x4 acc[MFW][NF];
  #pragma unroll
  for (int i = 0; i < MFW; ++i)
    #pragma unroll
    for (int j = 0; j < NF; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const uint32_t *sp = a.step_ptr + static_cast<long>(active ? wt : 0) * (a.nchunks + 1);
  const uint32_t step0 = uniform(sp[0]);
  const uint32_t row0 = uniform(a.item_ptr[active ? wt : 0]);
  const float4 *A = static_cast<const float4 *>(a.a) + lane;
  const uint32_t *IT = a.items + g;

  float4 ra[DEPTH][MFW];
  uint32_t roff[DEPTH];
  auto fetch = [&](int slot, uint32_t s) {
    roff[slot] = IT[(static_cast<long>(row0) + (s - step0)) * 4];
    #pragma unroll
    for (int i = 0; i < MFW; ++i) ra[slot][i] = A[(static_cast<long>(s) * MFW + i) * 64];
  };
  auto compute = [&](int slot) {
    float4 bv[NF];
    #pragma unroll
    for (int j = 0; j < NF; ++j) bv[j] = *reinterpret_cast<const float4 *>(lds + vb[j] + roff[slot]);
    #pragma unroll
    for (int j = 0; j < NF; ++j)
      #pragma unroll
      for (int i = 0; i < MFW; ++i) {
        const float4 av = ra[slot][i];
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av.x, bv[j].x, acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av.y, bv[j].y, acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av.z, bv[j].z, acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av.w, bv[j].w, acc[i][j], 0, 0, 0);
      }
  };

  int ch0, ch1;
  split_range(a, wg.split, ch0, ch1);
  Stager<4, 8> st;
  st.init(a, b);
  if (st.ok && ch0 < ch1) st.issue(a, ch0 * a.cc);
  for (int ch = ch0; ch < ch1; ++ch) {
    __syncthreads();  // every wave is done with the previous chunk
    if (st.ok) st.commit(lds, a);
    else stage_halo<4>(lds, a, b, ch * a.cc);
    __syncthreads();
    if (st.ok && ch + 1 < ch1) st.issue(a, (ch + 1) * a.cc);  // overlaps this chunk's MFMAs
    if (!active) continue;
    const uint32_t s_beg = uniform(sp[ch]), s_end = uniform(sp[ch + 1]);
    if (s_beg == s_end) continue;
    for (int d = 0; d < DEPTH; ++d) fetch(d, min(s_beg + d, s_end - 1));
    uint32_t s = s_beg;
    const uint32_t s_last = s_end - 1;
    for (; s + DEPTH <= s_end; s += DEPTH) {
      // Straight-line body: the refill is unconditional (clamped to the last
      // step, a harmless re-read) so the memory-wait counters stay exact.
      static_for<DEPTH>([&](auto dc) {
        constexpr int D = decltype(dc)::value;
        compute(D);
        fetch(D, min(s + D + DEPTH, s_last));
      });
    }
    static_for<DEPTH - 1>([&](auto dc) {
      constexpr int D = decltype(dc)::value;
      if (s + D < s_end) compute(D);
    });
  }
  if (a.splits > 1) {
    if (active) {
      SlotWalk sw;
      sw.init(a, lane & 15, 16);
#pragma unroll
      for (int j = 0; j < NF; ++j) {
        const Slot sl = slot_at(a, b, sw.t, sw.h, sw.w);
        sw.next(a);
#pragma unroll
        for (int i = 0; i < MFW; ++i)
          put_partial(a, sl, wt * 16 * MFW + 16 * i + 4 * g, wg.split, acc[i][j]);
      }
    }
    return;
  }
  if (NF == 4 && MFW <= 2 && a.qt * a.qh * a.qw == 1) {
    // No pooling: a lane's accumulator holds 4 consecutive filters of one
    // voxel slot, so the epilogue runs on registers and stores straight to
    // y (no LDS tile, no barriers).  Narrow tiles only: in the wider ones
    // the extra live registers would cost the second wave per SIMD.
    if (active) {
      float4 bb[MFW];
#pragma unroll
      for (int i = 0; i < MFW; ++i) bb[i] = load_bias4(a, wt * 16 * MFW + 16 * i + 4 * g);
      SlotWalk sw;
      sw.init(a, lane & 15, 16);
#pragma unroll
      for (int j = 0; j < NF; ++j) {
        const Slot sl = slot_at(a, b, sw.t, sw.h, sw.w);
        sw.next(a);
        if (!sl.valid) continue;
#pragma unroll
        for (int i = 0; i < MFW; ++i) {
          const int m0 = wt * 16 * MFW + 16 * i + 4 * g;
          if (m0 >= a.c_out) continue;
          const float4 raw = make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
          put4<float>(a, sl.out, m0, activate4<float>(a, sl.out, m0, raw, bb[i]));
        }
      }
    }
    return;
  }
  const int m_wg0 = wg.tg * a.wpw * 16 * MFW;
  __syncthreads();  // the halo is no longer needed: reuse LDS for the tile
  if (active) {
#pragma unroll
    for (int j = 0; j < NF; ++j)
#pragma unroll
      for (int i = 0; i < MFW; ++i) {
        const int col = wt * 16 * MFW - m_wg0 + 16 * i + 4 * g;
        *reinterpret_cast<f32x4 *>(lds + (16 * j + (lane & 15)) * a.tile_row + col * 4) = acc[i][j];
      }
  }
  __syncthreads();
  tile_store<float>(a, b, lds, m_wg0);
}

// ---------------------------------------------------------------------------
// Exact f32 KGS kernel: v_mfma_f32_4x4x1_16b_f32, one 4x4 kernel block of
// one group at one kept position per instruction, no zero padding.
//
// Layouts (measured on gfx950): block b = lane/4; A[i][0] of block b in lane
// 4b+i; B[0][j] in lane 4b+j; D[i][j] in lane 4b+j, element i.  With
// CBSZ = 4 every block multiplies the A column of block ABID, so one VGPR of
// A data holds 16 columns (4 groups x 4 channels of an item) and lane l
// computes 4 filters of voxel slot l.  A wave tile is the 4 kernel groups
// of 16 consecutive filters; its items are the union of their kept
// (channel block, position) pairs, each with a 4-bit mask of the groups
// that keep it, and only those groups' instructions are issued.
// ---------------------------------------------------------------------------

template <int ABID>
__device__ __forceinline__ f32x4 mfma441(float av, float bv, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_4x4x1f32(av, bv, c, 4, ABID, 0);
}

template <int SUB>
__global__ __launch_bounds__(256) void kgs_exact_f32_kernel(ConvArgs a) {
  extern __shared__ __align__(16) uint8_t lds[];
  const int lane = threadIdx.x & 63;
  const Wg wg = decode_wg(a);
  const int wt = uniform(wg.tg * a.wpw + (static_cast<int>(threadIdx.x) >> 6));
  const bool active = wt < a.wave_tiles;
  const Brick b = decode_brick(a, wg.brick);

  int vb[SUB];
  {
    SlotWalk sw;
    sw.init(a, lane, 64);
#pragma unroll
    for (int s = 0; s < SUB; ++s) {
      vb[s] = slot_lds(a, b, sw.t, sw.h, sw.w);
      sw.next(a);
    }
  }

  f32x4 acc[4][SUB];
  #pragma unroll
  for (int gi = 0; gi < 4; ++gi)
    #pragma unroll
    for (int s = 0; s < SUB; ++s) acc[gi][s] = f32x4{0.f, 0.f, 0.f, 0.f};

  const uint32_t *sp = a.step_ptr + static_cast<long>(active ? wt : 0) * (a.nchunks + 1);
  const float *A = static_cast<const float *>(a.a);

  // Software pipeline over the wave's items (as in the 16-bit item kernel):
  // the weight value, LDS offset and keep bits of item i+D are in flight
  // from global memory, and the B operands of item i+1 are read from LDS,
  // while the MFMAs of item i run.  The item stream of the split runs across
  // chunk boundaries with clamped indices; only B waits for a chunk's halo.
  constexpr int D = 8;
  float ra[D];
  uint32_t roff[D], rkeep[D];
  float4 rb[2][SUB];
  auto fetch = [&](int slot, uint32_t it) {
    ra[slot] = A[static_cast<long>(it) * 64 + lane];
    roff[slot] = a.items[it];
    rkeep[slot] = a.keep[it];
  };
  auto load_b = [&](int slot, uint32_t off) {
    #pragma unroll
    for (int s = 0; s < SUB; ++s) rb[slot][s] = *reinterpret_cast<const float4 *>(lds + vb[s] + off);
  };
  auto mma = [&](int bs, int as) {
    const uint32_t keep = uniform(rkeep[as]);
    const float av = ra[as];
    static_for<4>([&](auto gc) {
      constexpr int G = decltype(gc)::value;
      if (keep & (1u << G)) {
        #pragma unroll
        for (int s = 0; s < SUB; ++s) {
          acc[G][s] = mfma441<4 * G + 0>(av, rb[bs][s].x, acc[G][s]);
          acc[G][s] = mfma441<4 * G + 1>(av, rb[bs][s].y, acc[G][s]);
          acc[G][s] = mfma441<4 * G + 2>(av, rb[bs][s].z, acc[G][s]);
          acc[G][s] = mfma441<4 * G + 3>(av, rb[bs][s].w, acc[G][s]);
        }
      }
    });
  };

  int ch0, ch1;
  split_range(a, wg.split, ch0, ch1);
  const uint32_t S0 = uniform(sp[ch0]), S1 = uniform(sp[ch1]);
  const bool work = active && S1 > S0;
  const uint32_t LAST = work ? S1 - 1 : S0;
  Stager<4, 8> st;
  st.init(a, b);
  if (st.ok && ch0 < ch1) st.issue(a, ch0 * a.cc);
  if (work) {
#pragma unroll
    for (int d = 0; d < D; ++d) fetch(d, min(S0 + d, LAST));
  }
  for (int ch = ch0; ch < ch1; ++ch) {
    __syncthreads();  // every wave is done with the previous chunk
    if (st.ok) st.commit(lds, a);
    else stage_halo<4>(lds, a, b, ch * a.cc);
    __syncthreads();
    if (st.ok && ch + 1 < ch1) st.issue(a, (ch + 1) * a.cc);  // overlaps this chunk's MFMAs
    if (!work) continue;
    const uint32_t i_beg = uniform(sp[ch]), i_end = uniform(sp[ch + 1]);
    if (i_beg == i_end) continue;
    // Ring slots are relative to the chunk's first item: slot i % D for
    // weights, offsets and keep bits, i % 2 for B.
    load_b(0, uniform(roff[0]));
    uint32_t i = i_beg;
    for (; i + D <= i_end; i += D) {
      static_for<D>([&](auto dc) {
        constexpr int K = decltype(dc)::value;
        load_b((K + 1) & 1, uniform(roff[(K + 1) % D]));
        mma(K & 1, K);
        fetch(K, min(i + K + D, LAST));
        __builtin_amdgcn_sched_barrier(0);
      });
    }
    const uint32_t rem = i_end - i;  // tail: 0..D-1 items
    static_for<D - 1>([&](auto dc) {
      constexpr int K = decltype(dc)::value;
      if (K < rem) {
        if (K + 1 < rem) load_b((K + 1) & 1, uniform(roff[(K + 1) % D]));
        mma(K & 1, K);
        fetch(K, min(i + K + D, LAST));
      }
    });
    // The rings hold items i_end.. at slots (n + k) % D: rotate them to slot 0.
    const int n = static_cast<int>(i_end - i_beg);
    rotate_ring(ra, n % D);
    rotate_ring(roff, n % D);
    rotate_ring(rkeep, n % D);
  }
  if (a.splits > 1) {
    if (active) {
      SlotWalk sw;
      sw.init(a, lane, 64);
#pragma unroll
      for (int sb = 0; sb < SUB; ++sb) {
        const Slot sl = slot_at(a, b, sw.t, sw.h, sw.w);
        sw.next(a);
#pragma unroll
        for (int gi = 0; gi < 4; ++gi) put_partial(a, sl, wt * 16 + 4 * gi, wg.split, acc[gi][sb]);
      }
    }
    return;
  }
  const int m_wg0 = wg.tg * a.wpw * 16;
  __syncthreads();  // the halo is no longer needed: reuse LDS for the tile
  if (active) {
#pragma unroll
    for (int s = 0; s < SUB; ++s)
#pragma unroll
      for (int gi = 0; gi < 4; ++gi) {
        const int col = wt * 16 - m_wg0 + 4 * gi;
        *reinterpret_cast<f32x4 *>(lds + (64 * s + lane) * a.tile_row + col * 4) = acc[gi][s];
      }
  }
  __syncthreads();
  tile_store<float>(a, b, lds, m_wg0);
}

// ---------------------------------------------------------------------------
// Split reduction: y = act(sum over splits, in split order, + bias
// (+ residual)).  Fixed summation order keeps results run-to-run identical.
// ---------------------------------------------------------------------------

// Split reduction + epilogue (+ fused max-pool).  Each output (pooled voxel,
// four filters) gets wl x zl adjacent lanes: wl = window voxels (when the
// window has 2, 4, ... voxels; any other window is walked by one lane) and
// zl = lanes sharing the splits (split z goes to lane z mod zl, at most four
// per lane, all loads in flight together).  Lanes add their splits in
// increasing order, combine across the zl lanes by an xor butterfly (a fixed
// order, so every run gives the same bits), apply the epilogue per window
// voxel, and take the max across the wl lanes.  A block covers vpb pooled
// voxels x cpb filter quads; blockIdx.y picks the filter-quad range.
struct ReduceShape {
  int wl, zl, lpo, cpb, vpb, groups;
};

__host__ __device__ inline ReduceShape reduce_shape(const ConvArgs &a) {
  ReduceShape r;
  const int win = a.qt * a.qh * a.qw;
  r.wl = win > 1 && win <= 16 && (win & (win - 1)) == 0 ? win : 1;
  r.zl = 1;
  while (r.zl * 4 < a.splits && r.zl * 2 * r.wl <= 16) r.zl *= 2;
  r.lpo = r.wl * r.zl;  // divides 64
  r.groups = a.c_out4 >> 2;
  r.cpb = r.groups < 256 / r.lpo ? r.groups : 256 / r.lpo;
  r.vpb = 256 / (r.cpb * r.lpo);
  return r;
}

template <typename T>
__global__ __launch_bounds__(256) void reduce_splits_kernel(ConvArgs a) {
  const ReduceShape rs = reduce_shape(a);
  const int t = threadIdx.x;
  const DivMod u = divmod(t, rs.lpo), w = divmod(u.q, rs.cpb);
  const int z0 = u.r % rs.zl, e = u.r / rs.zl;
  const int c4 = static_cast<int>(blockIdx.y) * rs.cpb + w.r;
  const int pv = static_cast<int>(blockIdx.x) * rs.vpb + w.q;
  const int pvox_total = a.n * a.pto * a.pho * a.pwo;
  const bool live = w.q < rs.vpb && pv < pvox_total && c4 < rs.groups;
  const int m0 = 4 * c4;
  const DivMod x = divmod(live ? pv : 0, a.pwo), y = divmod(x.q, a.pho), z = divmod(y.q, a.pto);
  const int gw = x.r, gh = y.r, gt = z.r, nb = z.q;
  const long zstride = a.total_vox * a.c_out4;
  auto voxel = [&](int dt, int dh, int dw) {
    return ((static_cast<long>(nb) * a.to + gt * a.qt + dt) * a.ho + gh * a.qh + dh) * a.wo +
           gw * a.qw + dw;
  };
  // This lane's share of the split sum of voxel vox: splits z0, z0 + zl, ...
  auto partial = [&](long vox) {
    const float *p = a.ws + vox * a.c_out4 + m0;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int zz = z0; zz < a.splits; zz += 4 * rs.zl) {
      float4 v[4];
#pragma unroll
      for (int k = 0; k < 4; ++k)
        v[k] = zz + k * rs.zl < a.splits
                   ? *reinterpret_cast<const float4 *>(p + (zz + k * rs.zl) * zstride)
                   : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (zz + k * rs.zl < a.splits) acc = add4(acc, v[k]);
    }
    return acc;
  };
  auto across_splits = [&](float4 v) {
    for (int m = 1; m < rs.zl; m <<= 1) v = add4(v, shfl_xor4(v, m));
    return v;
  };
  const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
  const float4 bb = live ? load_bias4(a, m0) : zero;
  float4 best;
  if (rs.wl > 1) {
    const int dw = e % a.qw, dh = (e / a.qw) % a.qh, dt = e / (a.qw * a.qh);
    const long vox = voxel(dt, dh, dw);
    const float4 sum = across_splits(live ? partial(vox) : zero);
    best = live ? activate4<T>(a, vox, m0, sum, bb) : zero;
    for (int m = rs.zl; m < rs.lpo; m <<= 1) best = max4(best, shfl_xor4(best, m));
  } else {
    best = zero;
    for (int dt = 0; dt < a.qt; ++dt)  // uniform trip counts: shuffles stay converged
      for (int dh = 0; dh < a.qh; ++dh)
        for (int dw = 0; dw < a.qw; ++dw) {
          const long vox = voxel(dt, dh, dw);
          const float4 sum = across_splits(live ? partial(vox) : zero);
          const float4 v = live ? activate4<T>(a, vox, m0, sum, bb) : zero;
          best = (dt | dh | dw) ? max4(best, v) : v;
        }
  }
  if (live && u.r == 0 && m0 < a.c_out) put4<T>(a, pv, m0, best);
}

// ---------------------------------------------------------------------------
// 3-D max pooling, channels-last, no padding: one thread per output voxel
// and run of VEC channels.
// ---------------------------------------------------------------------------

struct PoolArgs {
  int n, c, t, h, w, kt, kh, kw, st, sh, sw, pt, ph, pw, to, ho, wo;
  int cv;       // channel vectors per voxel (c / VEC)
  int item0;    // first (voxel, channel vector) item of this launch
  int items;    // items of this launch (< 2^24)
};

// One thread per (output voxel, VEC-channel vector); channel vectors are
// the fastest index, so a wave reads and writes contiguous 16-byte runs.
// KT/KH/KW > 0: a compile-time window, unrolled so that all its loads are in
// flight together (from clamped, always valid addresses; positions outside
// the input are dropped at the max); 0: the window from the arguments.
template <typename T, int VEC, int KT, int KH, int KW>
__global__ __launch_bounds__(256) void maxpool_kernel(const T *__restrict__ x, T *__restrict__ y,
                                                      PoolArgs p) {
  const int item = static_cast<int>(blockIdx.x) * 256 + static_cast<int>(threadIdx.x);
  if (item >= p.items) return;
  const DivMod vc = divmod(item, p.cv);     // local item: < 2^24
  const int cb = vc.r;
  const int vox = vc.q + p.item0 / p.cv;    // item0 is a multiple of cv
  const DivMod a = divmod(vox, p.wo);
  const DivMod b = divmod(a.q, p.ho);
  const DivMod d = divmod(b.q, p.to);
  const int ow = a.r, oh = b.r, ot = d.r, nb = d.q;
  using Vec = std::conditional_t<VEC * sizeof(T) == 16, uint4, T>;
  union Pack { Vec u; T e[VEC]; };
  float best[VEC];
  bool any = false;
  for (int e = 0; e < VEC; ++e) best[e] = 0.f;
  auto take = [&](const Pack &v, bool ok) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const float f = static_cast<float>(v.e[e]);
      best[e] = ok && (!any || f > best[e]) ? f : best[e];
    }
    any = any || ok;
  };
  auto load = [&](int zt, int zh, int zw) {
    Pack v;
    const long vx = ((static_cast<long>(nb) * p.t + zt) * p.h + zh) * p.w + zw;
    v.u = *reinterpret_cast<const Vec *>(x + vx * p.c + cb * VEC);
    return v;
  };
  if constexpr (KT > 0) {
    Pack v[KT][KH][KW];
#pragma unroll
    for (int it = 0; it < KT; ++it)
#pragma unroll
      for (int ih = 0; ih < KH; ++ih)
#pragma unroll
        for (int iw = 0; iw < KW; ++iw)
          v[it][ih][iw] = load(min(max(ot * p.st - p.pt + it, 0), p.t - 1),
                               min(max(oh * p.sh - p.ph + ih, 0), p.h - 1),
                               min(max(ow * p.sw - p.pw + iw, 0), p.w - 1));
#pragma unroll
    for (int it = 0; it < KT; ++it)
#pragma unroll
      for (int ih = 0; ih < KH; ++ih)
#pragma unroll
        for (int iw = 0; iw < KW; ++iw) {
          const int zt = ot * p.st - p.pt + it, zh = oh * p.sh - p.ph + ih,
                    zw = ow * p.sw - p.pw + iw;
          take(v[it][ih][iw], zt >= 0 && zt < p.t && zh >= 0 && zh < p.h && zw >= 0 && zw < p.w);
        }
  } else {
    for (int it = 0; it < p.kt; ++it) {
      const int zt = ot * p.st - p.pt + it;
      if (zt < 0 || zt >= p.t) continue;
      for (int ih = 0; ih < p.kh; ++ih) {
        const int zh = oh * p.sh - p.ph + ih;
        if (zh < 0 || zh >= p.h) continue;
        for (int iw = 0; iw < p.kw; ++iw) {
          const int zw = ow * p.sw - p.pw + iw;
          if (zw < 0 || zw >= p.w) continue;
          take(load(zt, zh, zw), true);
        }
      }
    }
  }
  // (the host keeps padding at most half the window: every window holds
  // at least one input voxel, so `any` is set here)
  Pack o;
#pragma unroll
  for (int e = 0; e < VEC; ++e) o.e[e] = static_cast<T>(best[e]);
  *reinterpret_cast<Vec *>(y + static_cast<long>(vox) * p.c + cb * VEC) = o.u;
}

// ---------------------------------------------------------------------------
// Group norms and the reweighted group-lasso penalty (Section 4).
// A "unit" is what one norm covers: one kernel position of one kernel group
// (KGS) or a whole group (vanilla).  A workgroup owns filter group p and qb
// consecutive channel groups; in the [M][N][ks] weight tensor each of the
// group's g_m filter rows holds that block as one contiguous run of
// (channels x ks) elements, so the block is staged into LDS as fp32 with
// coalesced loads, every norm becomes a short sum over LDS, and the gradient
// and proximal outputs go back out in the same coalesced order.  Each unit
// is summed by one thread (KGS) or one wave with a fixed butterfly (vanilla),
// and the workgroup's penalty sum is a fixed tree: the results do not depend
// on timing.  The whole block is in LDS before anything is written, so the
// proximal output may overwrite the weights in place.
// ---------------------------------------------------------------------------

template <int NORM>
__device__ __forceinline__ float norm_term(float v) {
  return NORM == 2 ? v * v : fabsf(v);
}

template <typename T, int NORM, bool VANILLA>
__global__ __launch_bounds__(256) void group_reweight_kernel(GroupArgs a) {
  extern __shared__ __align__(16) float gl[];
  float *buf = gl;                        // [gme][len] staged weights
  float *unorm = gl + a.buf_elems;        // norm of each unit of the block
  float *ulp = unorm + a.unit_cap;        // lambda * penalty factor of each unit
  float *red = ulp + a.unit_cap;          // [256] penalty-sum reduction
  const int tid = static_cast<int>(threadIdx.x);
  const int blk = static_cast<int>(blockIdx.x);
  const int p = blk / a.nqc, qc = blk - p * a.nqc;
  const int m0 = p * a.gm, gme = min(a.gm, a.M - m0);
  const int c0 = qc * a.qb * a.gn, c1 = min(a.N, c0 + a.qb * a.gn);
  const int len = (c1 - c0) * a.ks;      // staged elements per filter row
  const int span = a.gn * a.ks;          // elements of one channel group in a row
  const int nq = (c1 - c0 + a.gn - 1) / a.gn;
  const int q0 = qc * a.qb;
  const T *src = static_cast<const T *>(a.w);
  const long row0 = static_cast<long>(m0) * a.N * a.ks + static_cast<long>(c0) * a.ks;
  const long pitch = static_cast<long>(a.N) * a.ks;  // elements between filter rows

  // Stage: tiles of 4 rows x 4 columns (o, o + 256, ...) per thread, so 16
  // loads are in flight before the LDS stores and each address is a row
  // base plus the column.
  for (int o0 = tid; o0 < len; o0 += 4 * 256) {
    for (int i0 = 0; i0 < gme; i0 += 4) {
      float v[4][4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const T *rp = src + row0 + static_cast<long>(min(i0 + r, gme - 1)) * pitch;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int o = o0 + 256 * c;
          v[r][c] = (i0 + r < gme && o < len) ? to_f32(rp[o]) : 0.f;
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int o = o0 + 256 * c;
          if (i0 + r < gme && o < len) buf[(i0 + r) * len + o] = v[r][c];
        }
    }
  }
  __syncthreads();

  float local = 0.f;  // this thread's share of sum(pen * norm)
  if constexpr (!VANILLA) {
    for (int u = tid; u < nq * a.ks; u += 256) {
      const DivMod d = divmod(u, a.ks);
      const int ql = d.q, pos = d.r;
      const int gne = min(a.gn, (c1 - c0) - ql * a.gn);
      float acc = 0.f;
      for (int i = 0; i < gme; ++i) {
        const float *col = buf + i * len + ql * span + pos;
        for (int j = 0; j < gne; ++j) acc += norm_term<NORM>(col[j * a.ks]);
      }
      const float n = NORM == 2 ? sqrtf(acc) : acc;
      const long gu = (static_cast<long>(p) * a.Q + q0 + ql) * a.ks + pos;
      const float pu = a.pen ? a.pen[gu] : 1.f;
      local += pu * n;
      if (a.norms) a.norms[gu] = n;
      if (a.pen_next) a.pen_next[gu] = 1.f / (n * n + a.eps);
      if (a.mask) a.mask[gu] = n > a.tau ? 1 : 0;
      unorm[u] = n;
      ulp[u] = a.lambda * pu;
    }
  } else {
    const int wave = tid >> 6, lane = tid & 63;
    for (int ql = wave; ql < nq; ql += 4) {
      const int cnt = min(a.gn, (c1 - c0) - ql * a.gn) * a.ks;  // contiguous per row
      float acc = 0.f;
      for (int i = 0; i < gme; ++i) {
        const float *run = buf + i * len + ql * span;
        for (int r = lane; r < cnt; r += 64) acc += norm_term<NORM>(run[r]);
      }
      // Butterfly: every lane ends with the same sum (each step adds the
      // same two values in either order).
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
      const float n = NORM == 2 ? sqrtf(acc) : acc;
      const long gq = static_cast<long>(p) * a.Q + q0 + ql;
      const float pu = a.pen ? a.pen[gq] : 1.f;
      if (lane == 0) {
        local += pu * n;
        if (a.norms) a.norms[gq] = n;
        if (a.pen_next) a.pen_next[gq] = 1.f / (n * n + a.eps);
        unorm[ql] = n;
        ulp[ql] = a.lambda * pu;
      }
      if (a.mask)
        for (int r = lane; r < a.ks; r += 64) a.mask[gq * a.ks + r] = n > a.tau ? 1 : 0;
    }
  }

  red[tid] = local;
  __syncthreads();  // also publishes unorm / ulp
  if (a.partial) {
    for (int off = 128; off > 0; off >>= 1) {
      if (tid < off) red[tid] += red[tid + off];
      __syncthreads();
    }
    if (tid == 0) a.partial[blk] = red[0];
  }

  if (a.grad || a.w_prox) {
    // Same 4 x 4 tiles: the unit of a column is the same in every row, and
    // a tile's gradient loads are all issued before its stores, so the
    // read-modify-write waits for memory once per tile.
    T *dst = static_cast<T *>(a.w_prox);
    for (int o0 = tid; o0 < len; o0 += 4 * 256) {
      float un[4], ul[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int o = min(o0 + 256 * c, len - 1);
        const DivMod e = divmod(o, span);
        const int u = VANILLA ? e.q : e.q * a.ks + divmod(e.r, a.ks).r;
        un[c] = unorm[u];
        ul[c] = ulp[u];
      }
      for (int i0 = 0; i0 < gme; i0 += 4) {
        float g0[4][4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const long rb = row0 + static_cast<long>(min(i0 + r, gme - 1)) * pitch;
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int o = o0 + 256 * c;
            g0[r][c] = (a.grad && i0 + r < gme && o < len) ? a.grad[rb + o] : 0.f;
          }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const long rb = row0 + static_cast<long>(min(i0 + r, gme - 1)) * pitch;
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int o = o0 + 256 * c;
            if (i0 + r >= gme || o >= len) continue;
            const float v = buf[(i0 + r) * len + o], n = un[c], lp = ul[c];
            const float sgn = v > 0.f ? 1.f : (v < 0.f ? -1.f : 0.f);
            if (a.grad)
              a.grad[rb + o] = g0[r][c] + (NORM == 2 ? (n > 0.f ? lp * v / n : 0.f) : lp * sgn);
            if (dst) {
              const float theta = a.step * lp;
              float z;
              if constexpr (NORM == 2) {
                const float f = n > 0.f ? 1.f - theta / n : 0.f;
                z = f > 0.f ? v * f : 0.f;
              } else {
                const float m = fabsf(v) - theta;
                z = m > 0.f ? sgn * m : 0.f;
              }
              dst[rb + o] = static_cast<T>(z);
            }
          }
        }
      }
    }
  }
}

// reg = lambda * the sum of the per-workgroup partial sums, in index order
// (a second launch: the kernel boundary makes every partial visible).
__global__ __launch_bounds__(256) void reg_finalize_kernel(const float *partial, int n,
                                                           float lambda, float *reg) {
  __shared__ float red[256];
  const int tid = static_cast<int>(threadIdx.x);
  float s = 0.f;
  for (int i = tid; i < n; i += 256) s += partial[i];
  red[tid] = s;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (tid < off) red[tid] += red[tid + off];
    __syncthreads();
  }
  if (tid == 0) *reg = lambda * red[0];
}

size_t halo_bytes(const ConvArgs &a) {
  const size_t halo = static_cast<size_t>(a.ht) * a.hh * a.hw * a.row;
  if (a.splits > 1) return halo;  // partials are stored from registers
  const size_t tile = static_cast<size_t>(16 * a.nf) * a.tile_row;  // epilogue tile: the slots
  return halo > tile ? halo : tile;
}

// Raise the kernel's dynamic LDS limit to the whole 160 KB once.
template <typename K>
hipError_t prepare(K kernel) {
  static std::atomic<bool> done{false};
  if (done.load(std::memory_order_acquire)) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  if (e == hipSuccess) done.store(true, std::memory_order_release);
  return e;
}

template <typename K>
int launch_conv(K kernel, const ConvArgs &a, void *stream) {
  const size_t lds = halo_bytes(a);
  const hipError_t e = prepare(kernel);
  if (e != hipSuccess) return e;
  const long blocks = a.grid > 0 ? a.grid : static_cast<long>(a.nbricks) * a.ntg * a.splits;
  if (blocks == 0) return hipSuccess;
  dim3 grid(static_cast<unsigned>(blocks));
  hipLaunchKernelGGL(kernel, grid, dim3(64 * a.wpw), lds, static_cast<hipStream_t>(stream), a);
  return hipGetLastError();
}

// Resident workgroups per CU for a kernel at an LDS size (0 when unknown).
template <typename K>
int resident(K kernel, size_t lds) {
  if (prepare(kernel) != hipSuccess) return 0;
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, reinterpret_cast<const void *>(kernel), 256,
                                                   lds) != hipSuccess)
    return 0;
  return n;
}

// Split-K scratch of the no-allocation forward entry point: every GPU the
// library runs on holds one copy for the life of the process.
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

}  // namespace

// Device address of this device's copy of `scratch`, looked up once per
// device with that device current (in host code the array's name is only a
// stand-in, never a device address).  NULL when the lookup fails.
void *noalloc_scratch() {
  constexpr int kMaxDev = 64;
  static std::mutex mu;
  static void *ptr[kMaxDev] = {};
  static bool looked[kMaxDev] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev) {
    (void)hipGetLastError();
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!looked[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) == hipSuccess) {
      ptr[dev] = p;
      looked[dev] = true;
    } else {
      (void)hipGetLastError();
    }
  }
  return ptr[dev];
}

int conv_resident(int variant, int dtype, int mfw, int nf, size_t lds) {
  switch (variant) {
    case kVarDenseItems16:
    case kVarKgsUnion16:
#define RT3D_RES16(T)                                                                  \
  do {                                                                                 \
    if (nf == 4) {                                                                     \
      if (mfw == 1) return resident(items16_kernel<T, 1, 4, true>, lds);               \
      if (mfw == 2) return resident(items16_kernel<T, 2, 4, true>, lds);               \
      if (mfw == 4) return resident(items16_kernel<T, 4, 4, true>, lds);               \
    } else {                                                                           \
      if (mfw == 1) return resident(items16_kernel<T, 1, 8, true>, lds);               \
      if (mfw == 2) return resident(items16_kernel<T, 2, 8, true>, lds);               \
      if (mfw == 4) return resident(items16_kernel<T, 4, 8, true>, lds);               \
    }                                                                                  \
  } while (0)
      if (dtype == RT3D_BF16) RT3D_RES16(__bf16);
      else RT3D_RES16(_Float16);
#undef RT3D_RES16
      return 0;
    case kVarKgsPair16:
      if (nf != 4) return 0;
      if (dtype == RT3D_BF16) {
        if (mfw == 1) return resident(items16_kernel<__bf16, 1, 4, true, 1>, lds);
        if (mfw == 2) return resident(items16_kernel<__bf16, 2, 4, true, 1>, lds);
        if (mfw == 4) return resident(items16_kernel<__bf16, 4, 4, true, 1>, lds);
        return 0;
      }
      if (mfw == 1) return resident(items16_kernel<_Float16, 1, 4, true, 1>, lds);
      if (mfw == 2) return resident(items16_kernel<_Float16, 2, 4, true, 1>, lds);
      if (mfw == 4) return resident(items16_kernel<_Float16, 4, 4, true, 1>, lds);
      return 0;
    case kVarKgsBlockPair16:
      if (nf != 4 || mfw != 1) return 0;
      if (dtype == RT3D_BF16) return resident(items16_kernel<__bf16, 1, 4, true, 2>, lds);
      return resident(items16_kernel<_Float16, 1, 4, true, 2>, lds);
    case kVarDenseItemsF32:
    case kVarKgsUnionF32:
      if (nf == 4) {
        if (mfw == 1) return resident(items_f32_kernel<1, 4>, lds);
        if (mfw == 2) return resident(items_f32_kernel<2, 4>, lds);
        if (mfw == 4) return resident(items_f32_kernel<4, 4>, lds);
      } else {
        if (mfw == 1) return resident(items_f32_kernel<1, 8>, lds);
        if (mfw == 2) return resident(items_f32_kernel<2, 8>, lds);
        if (mfw == 4) return resident(items_f32_kernel<4, 8>, lds);
      }
      return 0;
    case kVarKgsExactF32:
      return nf == 4 ? resident(kgs_exact_f32_kernel<1>, lds) : resident(kgs_exact_f32_kernel<2>, lds);
    default:
      return 0;
  }
}

size_t small_lds_bytes(const ConvArgs &a) {
  const size_t buf =
      ((static_cast<size_t>(a.ht) * a.hh * a.hw * 8 + 15) & ~static_cast<size_t>(15)) + 128;
  return 4 * 2 * buf;  // four waves, two halo buffers each (rows + a 2-byte sink slot per lane)
}

template <typename K>
int launch_small(K kernel, const ConvArgs &a, void *stream) {
  const hipError_t e = prepare(kernel);
  if (e != hipSuccess) return e;
  if (a.grid <= 0) return hipSuccess;
  hipLaunchKernelGGL(kernel, dim3(static_cast<unsigned>(a.grid)), dim3(256), small_lds_bytes(a),
                     static_cast<hipStream_t>(stream), a);
  return hipGetLastError();
}

#define RT3D_SMALL_EPL(T, M, S, FN, ...)                                                 \
  do {                                                                                   \
    if (epl2)                                                                            \
      return res ? FN((small_kernel<T, M, true, S, 2>), __VA_ARGS__)                     \
                 : FN((small_kernel<T, M, false, S, 2>), __VA_ARGS__);                   \
    return res ? FN((small_kernel<T, M, true, S, 4>), __VA_ARGS__)                       \
               : FN((small_kernel<T, M, false, S, 4>), __VA_ARGS__);                     \
  } while (0)
#define RT3D_SMALL_STEPS(T, M, FN, ...)                                                  \
  do {                                                                                   \
    if (steps8) RT3D_SMALL_EPL(T, M, 8, FN, __VA_ARGS__);                                \
    RT3D_SMALL_EPL(T, M, 4, FN, __VA_ARGS__);                                            \
  } while (0)
#define RT3D_SMALL_MFW(T, FN, ...)                                                       \
  do {                                                                                   \
    if (mfw == 1) RT3D_SMALL_STEPS(T, 1, FN, __VA_ARGS__);                               \
    if (mfw == 2) RT3D_SMALL_STEPS(T, 2, FN, __VA_ARGS__);                               \
  } while (0)
#define RT3D_SMALL_DISPATCH(FN, ...)                                                     \
  do {                                                                                   \
    const bool steps8 = a.steps_max > 4;                                                 \
    const bool epl2 = a.hw * a.c_in <= 127;                                              \
    const bool res = a.res != nullptr;                                                   \
    if (dtype == RT3D_BF16) RT3D_SMALL_MFW(__bf16, FN, __VA_ARGS__);                      \
    else RT3D_SMALL_MFW(_Float16, FN, __VA_ARGS__);                                      \
  } while (0)

int launch_small16(const ConvArgs &a, int dtype, int mfw, void *stream) {
  if (dtype != RT3D_BF16 && dtype != RT3D_F16) return hipErrorInvalidValue;
  RT3D_SMALL_DISPATCH(launch_small, a, stream);
  return hipErrorInvalidValue;
}

int small_resident(const ConvArgs &a, int dtype, int mfw) {
  const size_t lds = small_lds_bytes(a);
  RT3D_SMALL_DISPATCH(resident, lds);
  return 0;
}

int launch_items16(const ConvArgs &a, int dtype, int mfw, int map, void *stream) {
  const bool fast = a.c_in % 8 == 0 && a.x_pitch % 8 == 0 && a.x_off % 8 == 0;
  if (map == 2) {
    if (a.nf != 4 || mfw != 1) return hipErrorInvalidValue;
    if (dtype == RT3D_BF16)
      return fast ? launch_conv(items16_kernel<__bf16, 1, 4, true, 2>, a, stream)
                  : launch_conv(items16_kernel<__bf16, 1, 4, false, 2>, a, stream);
    if (dtype == RT3D_F16)
      return fast ? launch_conv(items16_kernel<_Float16, 1, 4, true, 2>, a, stream)
                  : launch_conv(items16_kernel<_Float16, 1, 4, false, 2>, a, stream);
    return hipErrorInvalidValue;
  }
  if (map == 1) {
    // 64-slot bricks only: with eight fragments the doubled B ring would
    // leave one wave per SIMD.
    if (a.nf != 4) return hipErrorInvalidValue;
#define RT3D_PAIR16(T, M)                                                                \
  do {                                                                                   \
    return fast ? launch_conv(items16_kernel<T, M, 4, true, 1>, a, stream)               \
                : launch_conv(items16_kernel<T, M, 4, false, 1>, a, stream);             \
  } while (0)
    if (dtype == RT3D_BF16) {
      if (mfw == 1) RT3D_PAIR16(__bf16, 1);
      if (mfw == 2) RT3D_PAIR16(__bf16, 2);
      if (mfw == 4) RT3D_PAIR16(__bf16, 4);
    } else if (dtype == RT3D_F16) {
      if (mfw == 1) RT3D_PAIR16(_Float16, 1);
      if (mfw == 2) RT3D_PAIR16(_Float16, 2);
      if (mfw == 4) RT3D_PAIR16(_Float16, 4);
    }
#undef RT3D_PAIR16
    return hipErrorInvalidValue;
  }
#define RT3D_ITEMS16(T, M)                                                         \
  do {                                                                             \
    if (a.nf == 4)                                                                 \
      return fast ? launch_conv(items16_kernel<T, M, 4, true>, a, stream)          \
                  : launch_conv(items16_kernel<T, M, 4, false>, a, stream);        \
    return fast ? launch_conv(items16_kernel<T, M, 8, true>, a, stream)            \
                : launch_conv(items16_kernel<T, M, 8, false>, a, stream);          \
  } while (0)
  if (a.nf != 4 && a.nf != 8) return hipErrorInvalidValue;
  if (dtype == RT3D_BF16) {
    if (mfw == 1) RT3D_ITEMS16(__bf16, 1);
    if (mfw == 2) RT3D_ITEMS16(__bf16, 2);
    if (mfw == 4) RT3D_ITEMS16(__bf16, 4);
  } else if (dtype == RT3D_F16) {
    if (mfw == 1) RT3D_ITEMS16(_Float16, 1);
    if (mfw == 2) RT3D_ITEMS16(_Float16, 2);
    if (mfw == 4) RT3D_ITEMS16(_Float16, 4);
  }
#undef RT3D_ITEMS16
  return hipErrorInvalidValue;
}

int launch_items_f32(const ConvArgs &a, int mfw, void *stream) {
  if (a.nf == 4) {
    if (mfw == 1) return launch_conv(items_f32_kernel<1, 4>, a, stream);
    if (mfw == 2) return launch_conv(items_f32_kernel<2, 4>, a, stream);
    if (mfw == 4) return launch_conv(items_f32_kernel<4, 4>, a, stream);
    return hipErrorInvalidValue;
  }
  if (a.nf != 8) return hipErrorInvalidValue;
  if (mfw == 1) return launch_conv(items_f32_kernel<1, 8>, a, stream);
  if (mfw == 2) return launch_conv(items_f32_kernel<2, 8>, a, stream);
  if (mfw == 4) return launch_conv(items_f32_kernel<4, 8>, a, stream);
  return hipErrorInvalidValue;
}

int launch_reduce_splits(const ConvArgs &a, int dtype, void *stream) {
  const ReduceShape rs = reduce_shape(a);
  const long pvox = static_cast<long>(a.n) * a.pto * a.pho * a.pwo;
  if (pvox == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((pvox + rs.vpb - 1) / rs.vpb),
                  static_cast<unsigned>((rs.groups + rs.cpb - 1) / rs.cpb));
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == RT3D_F32)
    hipLaunchKernelGGL(reduce_splits_kernel<float>, grid, dim3(256), 0, s, a);
  else if (dtype == RT3D_BF16)
    hipLaunchKernelGGL(reduce_splits_kernel<__bf16>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(reduce_splits_kernel<_Float16>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

int launch_kgs_exact_f32(const ConvArgs &a, void *stream) {
  if (a.nf == 4) return launch_conv(kgs_exact_f32_kernel<1>, a, stream);  // 64 slots: one per lane
  if (a.nf != 8) return hipErrorInvalidValue;
  return launch_conv(kgs_exact_f32_kernel<2>, a, stream);
}

// The windows of the C3D and S3D stacks get unrolled kernels.
template <typename T, int VEC>
void pool_launch(dim3 grid, hipStream_t s, const void *x, void *y, const PoolArgs &p) {
  const T *xs = static_cast<const T *>(x);
  T *ys = static_cast<T *>(y);
  auto win = [&](int a, int b, int c) { return p.kt == a && p.kh == b && p.kw == c; };
  if (win(3, 3, 3))
    hipLaunchKernelGGL((maxpool_kernel<T, VEC, 3, 3, 3>), grid, dim3(256), 0, s, xs, ys, p);
  else if (win(1, 3, 3))
    hipLaunchKernelGGL((maxpool_kernel<T, VEC, 1, 3, 3>), grid, dim3(256), 0, s, xs, ys, p);
  else if (win(2, 2, 2))
    hipLaunchKernelGGL((maxpool_kernel<T, VEC, 2, 2, 2>), grid, dim3(256), 0, s, xs, ys, p);
  else if (win(1, 2, 2))
    hipLaunchKernelGGL((maxpool_kernel<T, VEC, 1, 2, 2>), grid, dim3(256), 0, s, xs, ys, p);
  else
    hipLaunchKernelGGL((maxpool_kernel<T, VEC, 0, 0, 0>), grid, dim3(256), 0, s, xs, ys, p);
}

int launch_maxpool(int n, int c, int t, int h, int w, int kt, int kh, int kw, int st, int sh,
                   int sw, int pt, int ph, int pw, int to, int ho, int wo, int dtype,
                   const void *x, void *y, void *stream) {
  const long outs = static_cast<long>(n) * to * ho * wo;
  if (outs == 0 || c == 0) return hipSuccess;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int vec = dtype == RT3D_F32 ? (c % 4 == 0 ? 4 : 1) : (c % 8 == 0 ? 8 : 1);
  PoolArgs p{n, c, t, h, w, kt, kh, kw, st, sh, sw, pt, ph, pw, to, ho, wo, c / vec, 0, 0};
  // Launches of whole voxels with fewer than 2^24 items each (the fast
  // divide in the kernel needs that).
  const long per_launch = ((1l << 24) - 1) / p.cv * p.cv;
  const long total = outs * p.cv;
  for (long first = 0; first < total; first += per_launch) {
    p.item0 = static_cast<int>(first);
    p.items = static_cast<int>(std::min(per_launch, total - first));
    const dim3 grid(static_cast<unsigned>((p.items + 255) / 256));
    if (dtype == RT3D_F32) {
      if (vec == 4) pool_launch<float, 4>(grid, s, x, y, p);
      else pool_launch<float, 1>(grid, s, x, y, p);
    } else if (dtype == RT3D_BF16) {
      if (vec == 8) pool_launch<__bf16, 8>(grid, s, x, y, p);
      else pool_launch<__bf16, 1>(grid, s, x, y, p);
    } else {
      if (vec == 8) pool_launch<_Float16, 8>(grid, s, x, y, p);
      else pool_launch<_Float16, 1>(grid, s, x, y, p);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

int launch_group_reweight(const GroupArgs &a, int dtype, int norm, int scope, size_t lds,
                          void *stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 grid(static_cast<unsigned>(a.P) * static_cast<unsigned>(a.nqc));
#define RT3D_GROUP(T)                                                                        \
  do {                                                                                       \
    if (norm == 2 && scope == 0)                                                             \
      hipLaunchKernelGGL((group_reweight_kernel<T, 2, false>), grid, dim3(256), lds, s, a);  \
    else if (norm == 2)                                                                      \
      hipLaunchKernelGGL((group_reweight_kernel<T, 2, true>), grid, dim3(256), lds, s, a);   \
    else if (scope == 0)                                                                     \
      hipLaunchKernelGGL((group_reweight_kernel<T, 1, false>), grid, dim3(256), lds, s, a);  \
    else                                                                                     \
      hipLaunchKernelGGL((group_reweight_kernel<T, 1, true>), grid, dim3(256), lds, s, a);   \
  } while (0)
  if (dtype == RT3D_F32) RT3D_GROUP(float);
  else if (dtype == RT3D_BF16) RT3D_GROUP(__bf16);
  else RT3D_GROUP(_Float16);
#undef RT3D_GROUP
  return hipGetLastError();
}

int launch_reg_finalize(const float *partial, int n, float lambda, float *reg, void *stream) {
  hipLaunchKernelGGL(reg_finalize_kernel, dim3(1), dim3(256), 0, static_cast<hipStream_t>(stream),
                     partial, n, lambda, reg);
  return hipGetLastError();
}

}  // namespace rt3d
