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

#include <type_traits>
#include <utility>

#include "rt3d_internal.h"

namespace rt3d {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

template <int... Is, typename F>
__device__ __forceinline__ void static_for_impl(std::integer_sequence<int, Is...>, F &&f) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
  static_for_impl(std::make_integer_sequence<int, N>{}, f);
}

// ---------------------------------------------------------------------------
// Brick geometry
// ---------------------------------------------------------------------------

struct Brick {
  int nb;               // batch item
  int ot0, oh0, ow0;    // first output voxel of the brick
  int zt0, zh0, zw0;    // input coordinate of halo voxel (0, 0, 0)
};

__device__ __forceinline__ Brick decode_brick(const ConvArgs &a) {
  Brick b;
  int id = blockIdx.x;
  const int bwi = id % a.nbw;
  id /= a.nbw;
  const int bhi = id % a.nbh;
  id /= a.nbh;
  const int bti = id % a.nbt;
  b.nb = id / a.nbt;
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

__device__ __forceinline__ Slot decode_slot(const ConvArgs &a, const Brick &b, int s) {
  const int plane = a.bh * a.bw;
  int tt = s / plane;
  const int r = s - tt * plane;
  int hh = r / a.bw;
  int ww = r - hh * a.bw;
  Slot o;
  o.valid = tt < a.bt && b.ot0 + tt < a.to && b.oh0 + hh < a.ho && b.ow0 + ww < a.wo;
  if (!o.valid) tt = hh = ww = 0;
  o.lds = (((tt * a.st) * a.hh + hh * a.sh) * a.hw + ww * a.sw) * a.row;
  o.out = ((static_cast<long>(b.nb) * a.to + b.ot0 + tt) * a.ho + b.oh0 + hh) * a.wo + b.ow0 + ww;
  return o;
}

// Stage channels [c0, c0 + cc) of the input brick plus halo into LDS.
// Row r of the halo (one input voxel) holds cc channels, zero where the
// voxel is padding or the channel does not exist.
template <int ES>
__device__ __forceinline__ void stage_halo(uint8_t *lds, const ConvArgs &a, const Brick &b,
                                           int c0) {
  constexpr int EPP = 16 / ES;                 // elements per 16-byte piece
  const int ppr = a.cc / EPP;                  // pieces per halo row
  const int total = a.ht * a.hh * a.hw * ppr;
  const bool vec = (a.c_in % EPP) == 0;
  const uint8_t *xb = static_cast<const uint8_t *>(a.x);
  for (int idx = threadIdx.x; idx < total; idx += blockDim.x) {
    const int hv = idx / ppr;
    const int piece = idx - hv * ppr;
    const int xw = hv % a.hw;
    const int rest = hv / a.hw;
    const int xh = rest % a.hh;
    const int xt = rest / a.hh;
    const int zt = b.zt0 + xt, zh = b.zh0 + xh, zw = b.zw0 + xw;
    const int c = c0 + piece * EPP;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (zt >= 0 && zt < a.t && zh >= 0 && zh < a.h && zw >= 0 && zw < a.w && c < a.c_in) {
      const long vox = ((static_cast<long>(b.nb) * a.t + zt) * a.h + zh) * a.w + zw;
      const uint8_t *src = xb + (vox * a.c_in + c) * ES;
      if (vec) {
        v = *reinterpret_cast<const uint4 *>(src);
      } else {
        union {
          uint4 u;
          uint8_t bytes[16];
        } tmp;
        tmp.u = make_uint4(0, 0, 0, 0);
        const int n_el = min(EPP, a.c_in - c);
        for (int e = 0; e < n_el; ++e)
          for (int k = 0; k < ES; ++k) tmp.bytes[e * ES + k] = src[e * ES + k];
        v = tmp.u;
      }
    }
    *reinterpret_cast<uint4 *>(lds + hv * a.row + piece * 16) = v;
  }
}

// ---------------------------------------------------------------------------
// Epilogue: y = act(acc + bias (+ residual)), four consecutive filters of one
// voxel per call.
// ---------------------------------------------------------------------------

template <typename T>
__device__ __forceinline__ float to_f32(T v) { return static_cast<float>(v); }

template <typename T>
__device__ __forceinline__ void store4(const ConvArgs &a, long vox, int m0, float v0, float v1,
                                       float v2, float v3) {
  if (m0 >= a.c_out) return;
  float v[4] = {v0, v1, v2, v3};
  T *y = static_cast<T *>(a.y) + vox * a.c_out + m0;
  const T *res = a.res ? static_cast<const T *>(a.res) + vox * a.c_out + m0 : nullptr;
  if ((a.c_out & 3) == 0) {
    if (a.bias) {
      const float4 bb = *reinterpret_cast<const float4 *>(a.bias + m0);
      v[0] += bb.x; v[1] += bb.y; v[2] += bb.z; v[3] += bb.w;
    }
    if (res) {
      if constexpr (sizeof(T) == 4) {
        const float4 rr = *reinterpret_cast<const float4 *>(res);
        v[0] += rr.x; v[1] += rr.y; v[2] += rr.z; v[3] += rr.w;
      } else {
        union { uint2 u; T e[4]; } rr;
        rr.u = *reinterpret_cast<const uint2 *>(res);
        for (int r = 0; r < 4; ++r) v[r] += to_f32(rr.e[r]);
      }
    }
    if (a.relu)
      for (int r = 0; r < 4; ++r) v[r] = v[r] > 0.f ? v[r] : 0.f;
    if constexpr (sizeof(T) == 4) {
      *reinterpret_cast<float4 *>(y) = make_float4(v[0], v[1], v[2], v[3]);
    } else {
      union { uint2 u; T e[4]; } out;
      for (int r = 0; r < 4; ++r) out.e[r] = static_cast<T>(v[r]);
      *reinterpret_cast<uint2 *>(y) = out.u;
    }
  } else {
    for (int r = 0; r < 4 && m0 + r < a.c_out; ++r) {
      float x = v[r];
      if (a.bias) x += a.bias[m0 + r];
      if (res) x += to_f32(res[r]);
      if (a.relu) x = x > 0.f ? x : 0.f;
      y[r] = static_cast<T>(x);
    }
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
// Four waves share one brick; wave w computes wave tile blockIdx.y*4 + w:
// 16*MFW filters x 16*NF voxel slots.  Dense layers give every wave tile the
// full item list (and MFW > 1 shares each B fragment across filter rows);
// KGS layers give each 16-filter tile the union of the items its four kernel
// groups keep, with the pruned entries of that union stored as zero weights.
// ---------------------------------------------------------------------------

template <typename T, int MFW, int NF>
__global__ __launch_bounds__(256) void items16_kernel(ConvArgs a) {
  using V8 = std::conditional_t<std::is_same_v<T, __bf16>, bf16x8, f16x8>;
  extern __shared__ __align__(16) uint8_t lds[];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  const int wt = blockIdx.y * 4 + wave;
  const bool active = wt < a.wave_tiles;
  const Brick b = decode_brick(a);

  int vb[NF];
  for (int j = 0; j < NF; ++j) vb[j] = decode_slot(a, b, 16 * j + (lane & 15)).lds;

  f32x4 acc[MFW][NF];
  for (int i = 0; i < MFW; ++i)
    for (int j = 0; j < NF; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const uint32_t *sp = a.step_ptr + static_cast<long>(active ? wt : 0) * (a.nchunks + 1);
  const uint32_t step0 = sp[0];
  const uint32_t row0 = a.item_ptr[active ? wt : 0];
  const V8 *A = static_cast<const V8 *>(a.a);

  for (int ch = 0; ch < a.nchunks; ++ch) {
    __syncthreads();
    stage_halo<2>(lds, a, b, ch * a.cc);
    __syncthreads();
    if (!active) continue;
    const uint32_t s_end = sp[ch + 1];
    for (uint32_t s = sp[ch]; s < s_end; ++s) {
      const uint2 off = *reinterpret_cast<const uint2 *>(a.items + (static_cast<long>(row0) + (s - step0)) * 8 + 2 * g);
      V8 av[MFW];
      for (int i = 0; i < MFW; ++i) av[i] = A[(static_cast<long>(s) * MFW + i) * 64 + lane];
      for (int j = 0; j < NF; ++j) {
        const uint2 lo = *reinterpret_cast<const uint2 *>(lds + vb[j] + off.x);
        const uint2 hi = *reinterpret_cast<const uint2 *>(lds + vb[j] + off.y);
        const uint4 raw = make_uint4(lo.x, lo.y, hi.x, hi.y);
        const V8 bv = __builtin_bit_cast(V8, raw);
        for (int i = 0; i < MFW; ++i) {
          if constexpr (std::is_same_v<T, __bf16>)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[i], bv, acc[i][j], 0, 0, 0);
          else
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av[i], bv, acc[i][j], 0, 0, 0);
        }
      }
    }
  }
  if (!active) return;
  for (int j = 0; j < NF; ++j) {
    const Slot sl = decode_slot(a, b, 16 * j + (lane & 15));
    if (!sl.valid) continue;
    for (int i = 0; i < MFW; ++i) {
      const int m0 = wt * 16 * MFW + 16 * i + 4 * g;
      store4<T>(a, sl.out, m0, acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
    }
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
  extern __shared__ __align__(16) uint8_t lds[];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  const int wt = blockIdx.y * 4 + wave;
  const bool active = wt < a.wave_tiles;
  const Brick b = decode_brick(a);

  int vb[NF];
  for (int j = 0; j < NF; ++j) vb[j] = decode_slot(a, b, 16 * j + (lane & 15)).lds;

  f32x4 acc[MFW][NF];
  for (int i = 0; i < MFW; ++i)
    for (int j = 0; j < NF; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const uint32_t *sp = a.step_ptr + static_cast<long>(active ? wt : 0) * (a.nchunks + 1);
  const uint32_t step0 = sp[0];
  const uint32_t row0 = a.item_ptr[active ? wt : 0];
  const float4 *A = static_cast<const float4 *>(a.a);

  for (int ch = 0; ch < a.nchunks; ++ch) {
    __syncthreads();
    stage_halo<4>(lds, a, b, ch * a.cc);
    __syncthreads();
    if (!active) continue;
    const uint32_t s_end = sp[ch + 1];
    for (uint32_t s = sp[ch]; s < s_end; ++s) {
      const uint32_t off = a.items[(static_cast<long>(row0) + (s - step0)) * 4 + g];
      float4 av[MFW];
      for (int i = 0; i < MFW; ++i) av[i] = A[(static_cast<long>(s) * MFW + i) * 64 + lane];
      for (int j = 0; j < NF; ++j) {
        const float4 bv = *reinterpret_cast<const float4 *>(lds + vb[j] + off);
        for (int i = 0; i < MFW; ++i) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].x, bv.x, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].y, bv.y, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].z, bv.z, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].w, bv.w, acc[i][j], 0, 0, 0);
        }
      }
    }
  }
  if (!active) return;
  for (int j = 0; j < NF; ++j) {
    const Slot sl = decode_slot(a, b, 16 * j + (lane & 15));
    if (!sl.valid) continue;
    for (int i = 0; i < MFW; ++i) {
      const int m0 = wt * 16 * MFW + 16 * i + 4 * g;
      store4<float>(a, sl.out, m0, acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
    }
  }
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
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int wt = blockIdx.y * 4 + wave;
  const bool active = wt < a.wave_tiles;
  const Brick b = decode_brick(a);

  int vb[SUB];
  for (int s = 0; s < SUB; ++s) vb[s] = decode_slot(a, b, 64 * s + lane).lds;

  f32x4 acc[4][SUB];
  for (int gi = 0; gi < 4; ++gi)
    for (int s = 0; s < SUB; ++s) acc[gi][s] = f32x4{0.f, 0.f, 0.f, 0.f};

  const uint32_t *sp = a.step_ptr + static_cast<long>(active ? wt : 0) * (a.nchunks + 1);
  const float *A = static_cast<const float *>(a.a);

  for (int ch = 0; ch < a.nchunks; ++ch) {
    __syncthreads();
    stage_halo<4>(lds, a, b, ch * a.cc);
    __syncthreads();
    if (!active) continue;
    const uint32_t it_end = sp[ch + 1];
    for (uint32_t it = sp[ch]; it < it_end; ++it) {
      const uint32_t off = a.items[it];
      const uint32_t keep = a.keep[it];
      const float av = A[static_cast<long>(it) * 64 + lane];
      float4 bv[SUB];
      for (int s = 0; s < SUB; ++s) bv[s] = *reinterpret_cast<const float4 *>(lds + vb[s] + off);
      static_for<4>([&](auto gc) {
        constexpr int G = decltype(gc)::value;
        if (keep & (1u << G)) {
          for (int s = 0; s < SUB; ++s) {
            acc[G][s] = mfma441<4 * G + 0>(av, bv[s].x, acc[G][s]);
            acc[G][s] = mfma441<4 * G + 1>(av, bv[s].y, acc[G][s]);
            acc[G][s] = mfma441<4 * G + 2>(av, bv[s].z, acc[G][s]);
            acc[G][s] = mfma441<4 * G + 3>(av, bv[s].w, acc[G][s]);
          }
        }
      });
    }
  }
  if (!active) return;
  for (int s = 0; s < SUB; ++s) {
    const Slot sl = decode_slot(a, b, 64 * s + lane);
    if (!sl.valid) continue;
    for (int gi = 0; gi < 4; ++gi) {
      const int m0 = wt * 16 + 4 * gi;
      store4<float>(a, sl.out, m0, acc[gi][s][0], acc[gi][s][1], acc[gi][s][2], acc[gi][s][3]);
    }
  }
}

// ---------------------------------------------------------------------------
// 3-D max pooling, channels-last, no padding: one thread per output voxel
// and run of VEC channels.
// ---------------------------------------------------------------------------

template <typename T, int VEC>
__global__ __launch_bounds__(256) void maxpool_kernel(const T *__restrict__ x, T *__restrict__ y,
                                                      int n, int c, int t, int h, int w, int kt,
                                                      int kh, int kw, int st, int sh, int sw,
                                                      int to, int ho, int wo) {
  const long cv = c / VEC;
  const long total = static_cast<long>(n) * to * ho * wo * cv;
  for (long idx = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
       idx += static_cast<long>(gridDim.x) * blockDim.x) {
    const int cb = static_cast<int>(idx % cv);
    long r = idx / cv;
    const int ow = static_cast<int>(r % wo);
    r /= wo;
    const int oh = static_cast<int>(r % ho);
    r /= ho;
    const int ot = static_cast<int>(r % to);
    const long nb = r / to;
    float best[VEC];
    for (int e = 0; e < VEC; ++e) best[e] = -__builtin_huge_valf();
    for (int it = 0; it < kt; ++it)
      for (int ih = 0; ih < kh; ++ih)
        for (int iw = 0; iw < kw; ++iw) {
          const long vox = ((nb * t + ot * st + it) * h + oh * sh + ih) * w + ow * sw + iw;
          const T *src = x + vox * c + cb * VEC;
          for (int e = 0; e < VEC; ++e) {
            const float v = static_cast<float>(src[e]);
            best[e] = (v > best[e] || (it == 0 && ih == 0 && iw == 0)) ? v : best[e];
          }
        }
    T *dst = y + (((nb * to + ot) * ho + oh) * wo + ow) * c + cb * VEC;
    for (int e = 0; e < VEC; ++e) dst[e] = static_cast<T>(best[e]);
  }
}

size_t halo_bytes(const ConvArgs &a) { return static_cast<size_t>(a.ht) * a.hh * a.hw * a.row; }

template <typename K>
int launch_conv(K kernel, const ConvArgs &a, void *stream) {
  const size_t lds = halo_bytes(a);
  static bool attr_done = false;
  if (!attr_done) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr_done = true;
  }
  const long blocks_x = static_cast<long>(a.n) * a.nbt * a.nbh * a.nbw;
  const int blocks_y = (a.wave_tiles + 3) / 4;
  if (blocks_x == 0 || blocks_y == 0) return hipSuccess;
  dim3 grid(static_cast<unsigned>(blocks_x), static_cast<unsigned>(blocks_y));
  hipLaunchKernelGGL(kernel, grid, dim3(256), lds, static_cast<hipStream_t>(stream), a);
  return hipGetLastError();
}

}  // namespace

int launch_items16(const ConvArgs &a, int dtype, int mfw, void *stream) {
  if (dtype == RT3D_BF16) {
    if (mfw == 1) return launch_conv(items16_kernel<__bf16, 1, 8>, a, stream);
    if (mfw == 2) return launch_conv(items16_kernel<__bf16, 2, 8>, a, stream);
  } else if (dtype == RT3D_F16) {
    if (mfw == 1) return launch_conv(items16_kernel<_Float16, 1, 8>, a, stream);
    if (mfw == 2) return launch_conv(items16_kernel<_Float16, 2, 8>, a, stream);
  }
  return hipErrorInvalidValue;
}

int launch_items_f32(const ConvArgs &a, int mfw, void *stream) {
  if (mfw == 1) return launch_conv(items_f32_kernel<1, 8>, a, stream);
  if (mfw == 2) return launch_conv(items_f32_kernel<2, 8>, a, stream);
  return hipErrorInvalidValue;
}

int launch_kgs_exact_f32(const ConvArgs &a, void *stream) {
  return launch_conv(kgs_exact_f32_kernel<2>, a, stream);
}

int launch_maxpool(int n, int c, int t, int h, int w, int kt, int kh, int kw, int st, int sh,
                   int sw, int to, int ho, int wo, int dtype, const void *x, void *y,
                   void *stream) {
  const long outs = static_cast<long>(n) * to * ho * wo;
  if (outs == 0 || c == 0) return hipSuccess;
  hipStream_t s = static_cast<hipStream_t>(stream);
  auto grid_for = [&](long items) {
    long blocks = (items + 255) / 256;
    return static_cast<unsigned>(blocks < 65536 ? blocks : 65536);
  };
#define RT3D_POOL(T, VEC)                                                                      \
  hipLaunchKernelGGL((maxpool_kernel<T, VEC>), dim3(grid_for(outs * (c / VEC))), dim3(256), 0, s, \
                     static_cast<const T *>(x), static_cast<T *>(y), n, c, t, h, w, kt, kh, kw,   \
                     st, sh, sw, to, ho, wo)
  if (dtype == RT3D_F32) {
    if (c % 4 == 0) RT3D_POOL(float, 4); else RT3D_POOL(float, 1);
  } else if (dtype == RT3D_BF16) {
    if (c % 8 == 0) RT3D_POOL(__bf16, 8); else RT3D_POOL(__bf16, 1);
  } else {
    if (c % 8 == 0) RT3D_POOL(_Float16, 8); else RT3D_POOL(_Float16, 1);
  }
#undef RT3D_POOL
  return hipGetLastError();
}

}  // namespace rt3d
