// Internal definitions shared by the host planner and the HIP kernels of
// librt3d.  Not part of the public ABI.
#pragma once

#include <stdint.h>

#include "../../include/rt3d.h"

namespace rt3d {

constexpr uint64_t kMagic = 0x314b4e3344335452ull;  // "RT3D3NK1" little-endian
constexpr uint32_t kVersion = 3;
constexpr uint64_t kAlign = 256;                    // section alignment in a blob

// Kernel mappings (the `variant` field of rt3d_pack_info).
enum Variant : uint32_t {
  kVarDenseItems16 = 1,  // dense, 16x16x32 MFMA (bf16/f16), all (block, position) items
  kVarDenseItemsF32 = 2, // dense, 16x16x4 f32 MFMA
  kVarKgsUnion16 = 3,    // KGS, 16x16x32 MFMA over the union of a 16-filter tile's items
  kVarKgsExactF32 = 4,   // KGS, 4x4x1 f32 MFMA, exact per 4x4 kernel block
  kVarSmallDense16 = 5,  // dense, c_in <= 4: wave-private bricks, weights in registers
  kVarSmallKgs16 = 6,    // KGS, c_in <= 4: as above over the union of the wave tile's items
  kVarKgsPair16 = 7,     // KGS, 2:4 sparse 16x16x64 MFMA over pairs of items no group keeps
                         // both of; compact weight stream (kept 4x4 blocks only)
  kVarKgsBlockPair16 = 8,  // KGS, 2:4 sparse 16x16x64 MFMA over the channel-block pairs
                           // (2i, 2i+1) at one position, one 16-byte LDS read each
  kVarKgsUnionF32 = 9,   // KGS, 16x16x4 f32 MFMA over the union of a 16-filter tile's items
};

// Voxel tiling shared by every conv kernel: a workgroup computes a brick of
// bt x bh x bw output voxels of one batch item (64 voxel slots per wave
// step), staging the input brick plus halo for a chunk of `cc` channels in
// LDS with rows of `row` bytes per voxel.
struct Tiling {
  int32_t bt, bh, bw;      // output brick
  int32_t ht, hh, hw;      // halo extent in input voxels
  int32_t cc;              // channels per LDS chunk
  int32_t row;             // LDS bytes per halo voxel (cc * esize + pad)
  int32_t slots;           // voxel slots per workgroup (multiple of 64)
  int32_t nchunks;         // ceil(c_in / cc)
};

// Launch plan chosen at pack time, kept in rt3d_pack_info::plan (and hence
// in the blob header, which is a copy of the info struct).
struct Plan {
  Tiling tiling;
  int32_t mfw;             // 16-filter MFMA rows per wave tile
  int32_t wave_tiles;      // number of wave tiles
  int32_t items_per_step;  // items consumed per K-step
  int32_t tile_steps;      // most K-steps of one wave tile over all chunks
  int32_t gmap;            // kVarKgsUnion16: 1 if the keep section maps each wave tile's
                           // 4-filter block slots to the layer's blocks (u32 per slot)
  int32_t reserved;
  uint64_t step_ptr_off;   // u32 [wave_tiles][nchunks + 1]
  uint64_t item_ptr_off;   // u32 [wave_tiles]
  uint64_t items_off;      // u32 [...] LDS byte offset of each item
  uint64_t a_off;          // dtype [...], MFMA operand order
  uint64_t keep_off;       // u32 [...] (exact f32 variant: kept-group bits per item;
                           // pair variant: uint4 per step {keep, side, first block, 0};
                           // union variant with gmap: layer block of each tile slot)
};
static_assert(sizeof(Plan) <= sizeof(((rt3d_pack_info *)0)->plan), "plan does not fit");

// Everything a conv kernel needs, passed by value.
struct ConvArgs {
  const void *x;
  void *y;
  const void *res;
  const float *bias;
  const uint32_t *step_ptr;
  const uint32_t *item_ptr;
  const uint32_t *items;
  const uint32_t *keep;
  const uint32_t *gmap;  // layer 4-filter block of each wave-tile block slot, or NULL (identity)
  const void *a;
  int32_t n, c_in, c_out, t, h, w, to, ho, wo;
  int32_t st, sh, sw, pt, ph, pw;
  int32_t bt, bh, bw, nbt, nbh, nbw;
  int32_t ht, hh, hw, cc, row, nchunks;
  int32_t wave_tiles, relu;
  int32_t wpw;        // waves (wave tiles) per workgroup
  int32_t splits;     // channel-chunk splits (grid.z); > 1 writes fp32 partials to ws
  int32_t c_out4;     // c_out rounded up to 4 (partial row pitch)
  int32_t order;      // logical workgroup order: 0 = bricks fastest, 1 = filter tiles fastest
  long total_vox;     // n * to * ho * wo
  float *ws;          // [splits][total_vox][c_out4] partial sums (splits > 1)
  int32_t qt, qh, qw; // fused pooling window (1 = none)
  int32_t pto, pho, pwo;  // pooled output extent
  int32_t c_wg;       // filters per workgroup (wpw * 16 * mfw)
  int32_t tile_row;   // LDS bytes per voxel slot of the epilogue tile
  int32_t nbricks;    // n * nbt * nbh * nbw
  int32_t ntg;        // workgroups along the filters: ceil(wave_tiles / wpw)
  int32_t grid;       // workgroups launched (0: one per tile); fewer loop over tiles
  int32_t y_pitch;    // channels per voxel of y (>= c_out: fused concatenation)
  int32_t y_off;      // first channel of y this layer writes
  int32_t steps_max;  // most K-steps of one wave tile (the plan's tile_steps)
  int32_t x_pitch;    // channels per voxel of x (>= c_in: a slice of a wider tensor)
  int32_t x_off;      // first channel of x this layer reads
  int32_t nf;         // 16-slot voxel fragments per wave (slots / 16)
  int32_t a_bytes;    // bytes of the weight stream (pair variant: its buffer extent)
  int32_t gmap_slots; // entries of gmap (wave_tiles * 4 * mfw)
};

// Launch shape chosen at forward time from the batch size.
struct Launch {
  int wpw;
  int splits;
  uint64_t ws_bytes;
  int order;  // ConvArgs::order
};

// Group norms / reweighted group-lasso penalty (Section 4).  A workgroup owns
// filter group p and channel groups [qc*qb, qc*qb + qb) of one layer's
// [M][N][ks] weights; blockIdx.x = p * nqc + qc.
struct GroupArgs {
  const void *w;
  const float *pen;   // current penalty factor per unit, or NULL (all ones)
  float *norms;       // per unit, or NULL
  float *pen_next;    // per unit, or NULL
  float *partial;     // per workgroup sum of pen * norm, or NULL (no penalty value)
  float *grad;        // [M][N][ks] fp32, accumulated, or NULL
  uint8_t *mask;      // [P][Q][ks], or NULL
  void *w_prox;       // [M][N][ks] in the weight dtype, or NULL
  int32_t M, N, ks, gm, gn, P, Q;
  int32_t qb, nqc;    // channel groups per workgroup, workgroups per filter group
  int32_t buf_elems;  // LDS floats reserved for the staged block (gm * qb * gn * ks)
  int32_t unit_cap;   // LDS floats reserved per unit array (qb * ks, or qb for vanilla)
  float lambda, eps, tau, step;
};

// Bytes of the library's own split-K scratch (the no-allocation forward).
constexpr uint64_t kScratchBytes = 32ull << 20;
// Device address of the current device's scratch, NULL if it cannot be found.
void *noalloc_scratch();

// Kernel launchers (rt3d_kernels.hip).  Return hipSuccess or the launch error.
// Workgroups of the conv kernel for (variant, dtype, mfw, nf) that fit on one CU
// with `lds` bytes of dynamic LDS each; 0 when the runtime cannot say.
int conv_resident(int variant, int dtype, int mfw, int nf, size_t lds);
int launch_items16(const ConvArgs &a, int dtype, int mfw, int map, void *stream);
int launch_small16(const ConvArgs &a, int dtype, int mfw, void *stream);
size_t small_lds_bytes(const ConvArgs &a);
int small_resident(const ConvArgs &a, int dtype, int mfw);
int launch_items_f32(const ConvArgs &a, int mfw, void *stream);
int launch_kgs_exact_f32(const ConvArgs &a, void *stream);
int launch_reduce_splits(const ConvArgs &a, int dtype, void *stream);
int launch_group_reweight(const GroupArgs &a, int dtype, int norm, int scope, size_t lds,
                          void *stream);
int launch_reg_finalize(const float *partial, int n, float lambda, float *reg, void *stream);
int launch_maxpool(int n, int c, int t, int h, int w, int kt, int kh, int kw, int st, int sh,
                   int sw, int pt, int ph, int pw, int to, int ho, int wo, int dtype, const void *x,
                   void *y, void *stream);

}  // namespace rt3d
