// gfx950 (CDNA4) kernels of the batched Muon step.
//
// Per chunk of same-shape matrices (Sec. 6.6 shape fusion):
//   k_prologue   momentum update in place, per-tile sums of u^2, and X~ = u
//                (unscaled), transpose-first, cast; writes X~ and X~^T (HBM-bound)
//   k_finalize   r = 1 / (||u||_F + eps) per matrix (fixed-order sum)
//   k_rescale    X0 = r*u for the rare matrices whose r the first products
//                cannot apply (see k_finalize); others exit at once
//   k_gemm_tile  the three contractions of Eq. (1) on MFMA, 256 x 256 tiles
//                (bf16; S and L multiples of 256):
//                  A  = X X^T          (Gram, upper-triangle tiles only)
//                  B  = b A + c A A    (A is symmetric, so A A = A A^T)
//                  X' = a X + B X      (X read K-major by transposing LDS reads)
//                the last step's epilogue applies the update to W directly;
//   k_gemm_nt    the same on 128 x 128 tiles (fp32 NS and other extents;
//                writes mirrored A and B and reads X^T);
//   k_apply_x0   the update from X0 when K = 0;
//   k_adamw      AdamW for the parameters Muon does not take.
//
// All workspace buffers are zero-padded to multiples of 128 in both extents,
// so the contraction kernels never test bounds; zero padding is preserved by
// every step (padded rows/columns of X, A and B stay exactly zero).
#include <hip/hip_runtime.h>

#include <type_traits>
#include <utility>

#include "muon_internal.h"

namespace muon {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// bfloat16 storage: uint16 bit patterns.  Widening is exact; narrowing is
// the hardware conversion (v_cvt_pk_bf16_f32): round to nearest, ties to
// even, NaN stays NaN, overflow to infinity.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}
// lo | hi << 16, both rounded as above, in one instruction
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<uint16_t>(uint16_t v) { return bf16_to_f32(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ uint16_t from_f32<uint16_t>(float v) { return f32_to_bf16(v); }

__device__ __forceinline__ float load_as_f32(const void* p, int64_t i, int dt) {
  return dt == DT_BF16 ? bf16_to_f32(static_cast<const uint16_t*>(p)[i])
                       : static_cast<const float*>(p)[i];
}
__device__ __forceinline__ void store_from_f32(void* p, int64_t i, int dt, float v) {
  if (dt == DT_BF16) static_cast<uint16_t*>(p)[i] = f32_to_bf16(v);
  else static_cast<float*>(p)[i] = v;
}

// 8 consecutive elements at base + i (16-byte aligned) as fp32, and back
// (bf16 rounded to nearest even).
template <typename T>
__device__ __forceinline__ void load8(const T* base, int64_t i, float out[8]) {
  if constexpr (sizeof(T) == 2) {
    const u32x4_t raw = *reinterpret_cast<const u32x4_t*>(base + i);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      out[2 * q] = __uint_as_float(raw[q] << 16);
      out[2 * q + 1] = __uint_as_float(raw[q] & 0xffff0000u);
    }
  } else {
    const float4 a = *reinterpret_cast<const float4*>(base + i);
    const float4 b = *reinterpret_cast<const float4*>(base + i + 4);
    out[0] = a.x; out[1] = a.y; out[2] = a.z; out[3] = a.w;
    out[4] = b.x; out[5] = b.y; out[6] = b.z; out[7] = b.w;
  }
}

template <typename T>
__device__ __forceinline__ void store8(T* base, int64_t i, const float in[8]) {
  if constexpr (sizeof(T) == 2) {
    u32x4_t raw;
#pragma unroll
    for (int q = 0; q < 4; ++q) raw[q] = pack_bf16x2(in[2 * q], in[2 * q + 1]);
    *reinterpret_cast<u32x4_t*>(base + i) = raw;
  } else {
    *reinterpret_cast<float4*>(base + i) = make_float4(in[0], in[1], in[2], in[3]);
    *reinterpret_cast<float4*>(base + i + 4) = make_float4(in[4], in[5], in[6], in[7]);
  }
}

// Fixed-order sum over a 256-thread block: butterfly within each 64-lane
// wavefront, then the four wave sums in wave order.  Deterministic.  In fp64:
// the sums of u^2 stay finite for every finite u (|u| < 2^128 and at most
// 2^62 elements), where binary32 would overflow once |u| passes 2^64.
__device__ __forceinline__ double block_sum_256(double v, double* red4) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red4[wave] = v;
  __syncthreads();
  return ((red4[0] + red4[1]) + red4[2]) + red4[3];
}

// The factor r = 1 / (||u|| + eps) as two binary32 factors whose product is r
// (rounded once), each a normal number: r itself when it is one, else a power
// of two 2^-64 or 2^64 times the rest, for norms beyond 2^126 or below 2^-126.
__device__ __forceinline__ void split_scale(double r, float& s1, float& s2) {
  if (r < 0x1p-126 && r > 0.0) {
    s1 = 0x1p-64f;
    s2 = static_cast<float>(r * 0x1p64);
  } else if (r > 0x1p126) {
    s1 = 0x1p64f;
    s2 = static_cast<float>(r * 0x1p-64);
  } else {
    s1 = 1.0f;
    s2 = static_cast<float>(r);
  }
}

// ---------------------------------------------------------------------------
// Prologue, one pass over g and the momentum.  X0 = u / (||u|| + eps) needs
// the norm of all of u before any element of X0 can be formed; rather than
// reading g and the momentum a second time, this pass writes X~ = u unscaled
// (cast to the NS dtype) and the first Newton-Schulz step applies r = 1 /
// (||u|| + eps) to its products: A0 = r^2 (X~ X~^T), X1 = r (a X~ + B0 X~).
//
// A workgroup owns a 64x64 tile of the padded X extent (S x L), or a 32x128
// one when u is s x l and no X^T is kept (see tile_of).  It reads the
// matching tile of u's inputs row-wise, 8 consecutive elements per access
// (16-byte loads where the rows allow it, element by element at ragged
// edges), updates the momentum in place, writes X~ into whichever of X / X^T
// has u's layout (16-byte stores) and, through LDS, into the other (16-byte
// stores of 8 elements of one column), and stores its tile's sum of u^2 (a
// fixed-order reduction).  Zero outside the matrix.
// grid = (L/64, S/64, matrices).
// ---------------------------------------------------------------------------
template <typename XT>
struct TileStage {
  static constexpr int LDT = sizeof(XT) == 2 ? 66 : 65;  // LDS row stride (odd word stride)
};

// Tile (i0, j0) of X (origin in X coordinates) of matrix m: the same tile of
// u, its two destinations and their row strides.
template <typename XT>
struct TileDst {
  int ur0, uc0;
  XT* D;       // u's own layout (X when u is s x l, X^T when l x s), or null
  int ldD;
  XT* Tb;      // the transpose, through LDS, or null
  int ldT;
};

// Tile tt (row-major over the (S/64) x (L/64) grid) of matrix m.  A matrix
// with no transpose to write takes 32 x 128 tiles instead (the same count
// and the same 4096 elements each), whose 256-byte row pieces read and
// write more contiguously; `wide` says which.
template <typename XT>
__device__ __forceinline__ TileDst<XT> tile_dst(const MatDesc& md, const ChunkGeom& cg, int m, int i0, int j0,
                                                XT* X, XT* XTb);

template <typename XT>
__device__ __forceinline__ TileDst<XT> tile_of(const MatDesc& md, const ChunkGeom& cg, int m, int tt, XT* X,
                                               XT* XTb, bool& wide) {
  wide = md.transposed == 0 && XTb == nullptr;
  if (wide) {
    const int tx = cg.L / 128;
    return tile_dst(md, cg, m, (tt / tx) * 32, (tt % tx) * 128, X, XTb);
  }
  const int tx = cg.L / 64;
  return tile_dst(md, cg, m, (tt / tx) * 64, (tt % tx) * 64, X, XTb);
}

template <typename XT>
__device__ __forceinline__ TileDst<XT> tile_dst(const MatDesc& md, const ChunkGeom& cg, int m, int i0, int j0,
                                                XT* X, XT* XTb) {
  const bool tr = md.transposed != 0;
  const int64_t matX = static_cast<int64_t>(cg.S) * cg.L;
  XT* Xm = X + m * matX;
  XT* XTm = XTb ? XTb + m * matX : nullptr;
  TileDst<XT> t;
  t.ur0 = tr ? j0 : i0;
  t.uc0 = tr ? i0 : j0;
  t.D = tr ? XTm : Xm;
  t.ldD = tr ? cg.S : cg.L;
  t.Tb = tr ? Xm : XTm;
  t.ldT = tr ? cg.L : cg.S;
  return t;
}

// Phase 2 of a tile: rows of the transpose out of LDS, 16 bytes a thread.
template <typename XT>
__device__ __forceinline__ void write_transposed(const XT* tile, const TileDst<XT>& t) {
  constexpr int LDT = TileStage<XT>::LDT;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int c = threadIdx.x + 256 * k;          // row c / 8 of the transpose, 8 (c % 8) ..
    const int trow = c >> 3, r8 = (c & 7) * 8;
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = to_f32<XT>(tile[(r8 + q) * LDT + trow]);
    store8(t.Tb, static_cast<int64_t>(t.uc0 + trow) * t.ldT + t.ur0 + r8, v);
  }
}

// One tile of the prologue (UPDATE_MOM: advance the momentum and write it
// back; otherwise the momentum has been advanced already).  Returns this
// thread's sum of u^2 (fp64).  out = (u * s1) * s2.
template <typename GT, typename XT, bool MOM, bool UPDATE_MOM, bool WIDE>
__device__ __forceinline__ double prologue_tile(const MatDesc& md, const StepScalars& sc, const TileDst<XT>& t,
                                                float s1, float s2, XT* tile) {
  constexpr int LDT = TileStage<XT>::LDT;
  constexpr int CPR = WIDE ? 16 : 8;              // 8-element chunks per tile row
  const GT* __restrict__ g = static_cast<const GT*>(md.g);
  const float beta = sc.beta, omb = sc.one_minus_beta;
  double acc = 0.0;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int c = threadIdx.x + 256 * k;          // chunk: row c / CPR, columns 8 (c % CPR) ..
    const int row = c / CPR, col = (c % CPR) * 8;
    const int ur = t.ur0 + row, uc = t.uc0 + col;
    float v[8];
    if (md.row8_ok && ur < md.rows && uc + 8 <= md.cols) {
      float gv[8], bv[8];
      load8(g, view_index(md, ur, uc), gv);
      if (MOM) {
        const int64_t ib = buf_index(md, ur, uc);
        load8(md.buf, ib, bv);
        if (UPDATE_MOM) {
#pragma unroll
          for (int q = 0; q < 8; ++q) bv[q] = fmaf(beta, bv[q], omb * gv[q]);
          store8(md.buf, ib, bv);
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = sc.nesterov ? fmaf(beta, bv[q], omb * gv[q]) : bv[q];
      } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = gv[q];
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        acc = fma(static_cast<double>(v[q]), static_cast<double>(v[q]), acc);
        v[q] = (v[q] * s1) * s2;
      }
    } else {  // padding stays exactly zero, whatever the scale
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        v[q] = 0.f;
        if (ur < md.rows && uc + q < md.cols) {
          const float gv = to_f32<GT>(g[view_index(md, ur, uc + q)]);
          if (MOM) {
            const int64_t ib = buf_index(md, ur, uc + q);
            float bn = md.buf[ib];
            if (UPDATE_MOM) {
              bn = fmaf(beta, bn, omb * gv);
              md.buf[ib] = bn;
            }
            v[q] = sc.nesterov ? fmaf(beta, bn, omb * gv) : bn;
          } else {
            v[q] = gv;
          }
          acc = fma(static_cast<double>(v[q]), static_cast<double>(v[q]), acc);
          v[q] = (v[q] * s1) * s2;
        }
      }
    }
    if (t.D) store8(t.D, static_cast<int64_t>(ur) * t.ldD + uc, v);
    if (!WIDE && t.Tb) {
#pragma unroll
      for (int q = 0; q < 8; ++q) tile[row * LDT + col + q] = from_f32<XT>(v[q]);
    }
  }
  return acc;
}

template <typename GT, typename XT, bool MOM>
__global__ __launch_bounds__(256) void k_prologue(const MatDesc* __restrict__ desc, StepScalars sc, ChunkGeom cg,
                                                  XT* __restrict__ X, XT* __restrict__ XTb,
                                                  double* __restrict__ partials) {
  __shared__ XT tile[64 * TileStage<XT>::LDT];
  __shared__ double red4[4];
  const int m = blockIdx.z;
  const MatDesc md = desc[m];
  bool wide;
  const TileDst<XT> t = tile_of(md, cg, m, blockIdx.y * gridDim.x + blockIdx.x, X, XTb, wide);
  const double acc = wide ? prologue_tile<GT, XT, MOM, true, true>(md, sc, t, 1.f, 1.f, tile)
                          : prologue_tile<GT, XT, MOM, true, false>(md, sc, t, 1.f, 1.f, tile);
  const double s = block_sum_256(acc, red4);  // (its barrier also publishes the LDS tile)
  if (threadIdx.x == 0)
    partials[static_cast<int64_t>(m) * (gridDim.x * gridDim.y) + blockIdx.y * gridDim.x + blockIdx.x] = s;
  if (!t.Tb) return;  // uniform over the block
  __syncthreads();
  write_transposed(tile, t);
}

// r = 1 / (sqrt(sum of partials) + eps), one workgroup per matrix, in fp64,
// and the scale the first products apply: r itself while X~ X~^T stays well
// inside the fp32 range (||u|| between 2^-40 and 2^40), else 1 (k_rescale
// then writes r*u into X instead).  1024 threads each sum every 1024th
// partial into four accumulators (independent loads in flight; an 8192 x
// 28672 matrix has 57344 partials), combined in a fixed order.
__global__ __launch_bounds__(1024) void k_finalize(const double* __restrict__ partials, int nparts, float eps,
                                                   double* __restrict__ rscale, float* __restrict__ xscale) {
  __shared__ double red16[16];
  const int m = blockIdx.x;
  const double* p = partials + static_cast<int64_t>(m) * nparts;
  double a[4] = {0.0, 0.0, 0.0, 0.0};
  int i = threadIdx.x;
  for (; i + 3 * 1024 < nparts; i += 4 * 1024) {
#pragma unroll
    for (int q = 0; q < 4; ++q) a[q] += p[i + q * 1024];
  }
  if (i < nparts) a[0] += p[i];
  if (i + 1024 < nparts) a[1] += p[i + 1024];
  if (i + 2048 < nparts) a[2] += p[i + 2048];
  double v = (a[0] + a[1]) + (a[2] + a[3]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  if ((threadIdx.x & 63) == 0) red16[threadIdx.x >> 6] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int w = 0; w < 16; ++w) s += red16[w];
  if (threadIdx.x == 0) {
    const double r = 1.0 / (sqrt(s) + static_cast<double>(eps));
    rscale[m] = r;
    xscale[m] = (r >= 0x1p-40 && r <= 0x1p40) ? static_cast<float>(r) : 1.0f;  // NaN fails both tests
  }
}

// X0 = r*u, written over X~, for the matrices whose scale k_finalize left at
// 1 (a norm outside the range above, zero with eps = 0, or NaN); every other
// matrix's workgroups return at once.  The momentum is already advanced.
// grid = (workgroups per matrix, matrices); each loops over its tiles.
template <typename GT, typename XT, bool MOM>
__global__ __launch_bounds__(256) void k_rescale(const MatDesc* __restrict__ desc, const double* __restrict__ rscale,
                                                 const float* __restrict__ xscale, StepScalars sc, ChunkGeom cg,
                                                 XT* __restrict__ X, XT* __restrict__ XTb) {
  __shared__ XT tile[64 * TileStage<XT>::LDT];
  const int m = blockIdx.y;
  const double r = rscale[m];
  if (xscale[m] != 1.0f || r == 1.0) return;  // uniform over the block
  float s1, s2;
  split_scale(r, s1, s2);
  const MatDesc md = desc[m];
  const int ntiles = (cg.L / 64) * (cg.S / 64);
  for (int tt = blockIdx.x; tt < ntiles; tt += gridDim.x) {
    bool wide;
    const TileDst<XT> t = tile_of(md, cg, m, tt, X, XTb, wide);
    if (wide) (void)prologue_tile<GT, XT, MOM, false, true>(md, sc, t, s1, s2, tile);
    else (void)prologue_tile<GT, XT, MOM, false, false>(md, sc, t, s1, s2, tile);
    if (t.Tb) {  // uniform over the block
      __syncthreads();
      write_transposed(tile, t);
      __syncthreads();  // the next tile overwrites the LDS tile
    }
  }
}

// ---------------------------------------------------------------------------
// C = P Q^T on MFMA, P: M x K and Q: N x K row-major (K contiguous), all
// extents multiples of 128.  256 threads = 4 wavefronts in a 2 x 2 grid,
// each owning a 64 x 64 sub-tile = 2 x 2 blocks of the 32x32 MFMA.  K is
// staged through LDS 128 bytes per row at a time (64 bf16 or 32 fp32),
// double-buffered, with the next slab prefetched into registers while the
// current one is multiplied.
//
// bf16: v_mfma_f32_32x32x16_bf16, a lane supplies 8 consecutive k of its row.
// fp32: v_mfma_f32_32x32x2_f32, a lane holds 4 consecutive k and issues four
//       MFMAs (lanes 0-31 give k = j, lanes 32-63 give k = 4 + j).
// In both, a lane's operand for a 32-k (bf16) / 8-k (fp32) group is the 16
// bytes at byte offset 16*(lane/32) of the group, so the LDS geometry is the
// same for both element types.
//
// Output layout of a 32x32 block: lane l, register r holds
//   row 8*(r/4) + 4*(l/32) + (r%4), column l%32.
// ---------------------------------------------------------------------------
enum Epi : int { EPI_GRAM = 0, EPI_POLY = 1, EPI_UPDATE = 2, EPI_FINAL = 3,
                 // final-step variants of the 256-tile kernel: update W / write out, bf16 / fp32
                 EPI_FINAL_W_BF16 = 4, EPI_FINAL_W_F32 = 5, EPI_FINAL_O_BF16 = 6, EPI_FINAL_O_F32 = 7 };

struct GemmArgs {
  const char* P;   int64_t p_mat;  int32_t ldp;   // bytes
  const char* Q;   int64_t q_mat;  int32_t ldq;
  int32_t k_slabs;                               // K * elem / 128
  int32_t tiles_m, tiles_n, syrk, tiles_per_mat;
  const char* E;   int64_t e_mat;  int32_t lde;   // epilogue input (A or X), bytes
  const char* ET;  int64_t et_mat; int32_t ldet;  // the same values, transposed layout
  char* C;         int64_t c_mat;  int32_t ldc;   // output, direct orientation
  char* CT;        int64_t ct_mat; int32_t ldct;  // output, transposed orientation
  float alpha, beta;
  const MatDesc* desc;
  int32_t final_kind, param_dtype;
  int32_t s, l;
  int32_t total_tiles;                           // tiles_per_mat * matrices
  // operand storage, 256 x 256 kernel only: 0 row-major over K; 1 symmetric,
  // upper-triangle 256 x 256 tiles only; 2 (Q) stored K x N
  int32_t p_mode, q_mode;
  // 256 x 256 kernel, polynomial product: the A term is added to the
  // accumulators in the main loop (weight alpha = b/c, output beta * acc)
  // instead of being read again in the epilogue.  The update products
  // always add their a*X term that way on this kernel.
  int32_t e_loop;
  // First Newton-Schulz step: X holds X~ = u unscaled, and the product is
  // scaled per matrix by xscale (the Gram product by its square); null after.
  const float* xscale;
};

constexpr int kRowBytes = 144;                   // 128 data + 16 pad per LDS row
constexpr int kOpBytes = kTile * kRowBytes;      // one operand slab
constexpr int kStageBytes = 2 * kOpBytes;
constexpr int kFStride = 137;                    // fp32 epilogue tile stride (odd)
static_assert(kTile * kFStride * 4 <= 2 * kStageBytes, "epilogue tile fits in LDS");

template <typename T> struct Mma;
template <> struct Mma<uint16_t> {
  __device__ __forceinline__ static void run(const u32x4_t& a, const u32x4_t& b, f32x16_t& c) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
  }
};
template <> struct Mma<float> {
  __device__ __forceinline__ static void run(const u32x4_t& a, const u32x4_t& b, f32x16_t& c) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[j]), __uint_as_float(b[j]), c,
                                               0, 0, 0);
  }
};

template <typename T, int EPI>
__global__ __launch_bounds__(256, 2) void k_gemm_nt(GemmArgs ga) {
  __shared__ __attribute__((aligned(16))) char smem[2 * kStageBytes];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // ---- tile assignment -----------------------------------------------------
  const int mat = blockIdx.x / ga.tiles_per_mat;
  int t = blockIdx.x - mat * ga.tiles_per_mat;
  int bm, bn;
  if (ga.syrk) {  // upper-triangle tiles bm <= bn, row by row
    bm = 0;
    while (t >= ga.tiles_m - bm) { t -= ga.tiles_m - bm; ++bm; }
    bn = bm + t;
  } else {
    bm = t / ga.tiles_n;
    bn = t - bm * ga.tiles_n;
  }
  const char* Pb = ga.P + mat * ga.p_mat + static_cast<int64_t>(bm) * kTile * ga.ldp;
  const char* Qb = ga.Q + mat * ga.q_mat + static_cast<int64_t>(bn) * kTile * ga.ldq;

  // ---- main loop -----------------------------------------------------------
  // Global -> register staging: row (tid/8 + 32v), 16-byte column (tid%8).
  const int lrow = tid >> 3, lcol = (tid & 7) * 16;
  u32x4_t rp[4], rq[4];
  auto gload = [&](int ks) {
    const int64_t koff = static_cast<int64_t>(ks) * 128 + lcol;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      rp[v] = *reinterpret_cast<const u32x4_t*>(Pb + static_cast<int64_t>(lrow + 32 * v) * ga.ldp + koff);
      rq[v] = *reinterpret_cast<const u32x4_t*>(Qb + static_cast<int64_t>(lrow + 32 * v) * ga.ldq + koff);
    }
  };
  auto sstore = [&](int stage) {
    char* sp = smem + stage * kStageBytes;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      *reinterpret_cast<u32x4_t*>(sp + (lrow + 32 * v) * kRowBytes + lcol) = rp[v];
      *reinterpret_cast<u32x4_t*>(sp + kOpBytes + (lrow + 32 * v) * kRowBytes + lcol) = rq[v];
    }
  };

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int arow = wm * 64 + (lane & 31), brow = wn * 64 + (lane & 31);
  const int khalf = (lane >> 5) * 16;

  gload(0);
  sstore(0);
  __syncthreads();
  for (int ks = 0; ks < ga.k_slabs; ++ks) {
    const int stage = ks & 1;
    if (ks + 1 < ga.k_slabs) gload(ks + 1);
    const char* sp = smem + stage * kStageBytes;
#pragma unroll
    for (int grp = 0; grp < 4; ++grp) {
      u32x4_t a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = *reinterpret_cast<const u32x4_t*>(sp + (arow + 32 * i) * kRowBytes + grp * 32 + khalf);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        b[j] = *reinterpret_cast<const u32x4_t*>(sp + kOpBytes + (brow + 32 * j) * kRowBytes + grp * 32 + khalf);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) Mma<T>::run(a[i], b[j], acc[i][j]);
    }
    if (ks + 1 < ga.k_slabs) sstore(stage ^ 1);
    __syncthreads();
  }

  // ---- epilogue: accumulators -> LDS fp32 tile ------------------------------
  // On the first step the products are of X~ = u: the Gram tile is scaled
  // by r^2, the update's product and its a*X term by r.
  float s_acc = 1.f, s_e = 1.f;
  if (ga.xscale && EPI != EPI_POLY) {
    const float r = ga.xscale[mat];
    s_acc = EPI == EPI_GRAM ? r * r : r;
    s_e = r;
  }
  float* ft = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int col = wn * 64 + j * 32 + (lane & 31);
        ft[row * kFStride + col] = acc[i][j][r] * s_acc;
      }
  __syncthreads();

  const bool diag = ga.syrk && bm == bn;
  const int gi0 = bm * kTile, gj0 = bn * kTile;  // tile origin (rows of P, rows of Q)
  const MatDesc* md = (EPI == EPI_FINAL) ? ga.desc + mat : nullptr;
  const bool tr = (EPI == EPI_FINAL) ? md->transposed != 0 : false;

  // Phase A: direct orientation, consecutive lanes on consecutive columns.
  for (int idx = tid; idx < kTile * kTile; idx += 256) {
    const int r = idx >> 7, c = idx & 127;
    const int gi = gi0 + r, gj = gj0 + c;
    float v;
    if (EPI == EPI_GRAM || EPI == EPI_POLY) {
      v = diag && r > c ? ft[c * kFStride + r] : ft[r * kFStride + c];
      if (EPI == EPI_POLY) {
        const float e = to_f32<T>(*reinterpret_cast<const T*>(ga.E + mat * ga.e_mat + static_cast<int64_t>(gi) * ga.lde + gj * static_cast<int>(sizeof(T))));
        v = fmaf(ga.alpha, e, ga.beta * v);
      }
      const T o = from_f32<T>(v);
      *reinterpret_cast<T*>(ga.C + mat * ga.c_mat + static_cast<int64_t>(gi) * ga.ldc + gj * static_cast<int>(sizeof(T))) = o;
      if (!diag) ft[r * kFStride + c] = to_f32<T>(o);  // for the mirror store
    } else {
      const float e = to_f32<T>(*reinterpret_cast<const T*>(ga.E + mat * ga.e_mat + static_cast<int64_t>(gi) * ga.lde + gj * static_cast<int>(sizeof(T))));
      v = fmaf(ga.alpha * s_e, e, ft[r * kFStride + c]);
      if (EPI == EPI_UPDATE) {
        const T o = from_f32<T>(v);
        *reinterpret_cast<T*>(ga.C + mat * ga.c_mat + static_cast<int64_t>(gi) * ga.ldc + gj * static_cast<int>(sizeof(T))) = o;
        ft[r * kFStride + c] = to_f32<T>(o);
      } else {  // EPI_FINAL
        if (!tr) {
          if (gi < ga.s && gj < ga.l) {
            const int64_t pidx = view_index(*md, gi, gj);
            if (ga.final_kind == 0) {
              const float w = load_as_f32(md->W, pidx, ga.param_dtype);
              store_from_f32(md->W, pidx, ga.param_dtype, fmaf(md->decay, w, -md->upd_scale * v));
            } else {
              store_from_f32(md->out, pidx, ga.param_dtype, v);
            }
          }
        } else {
          ft[r * kFStride + c] = v;
        }
      }
    }
  }
  const bool phase_b = (EPI == EPI_GRAM || EPI == EPI_POLY) ? !diag : (EPI == EPI_UPDATE ? true : tr);
  if (!phase_b) return;  // uniform across the workgroup
  __syncthreads();
  // Phase B: transposed orientation, consecutive lanes on consecutive rows r.
  for (int idx = tid; idx < kTile * kTile; idx += 256) {
    const int c = idx >> 7, r = idx & 127;
    const float v = ft[r * kFStride + c];
    const int gi = gi0 + r, gj = gj0 + c;
    if (EPI == EPI_FINAL) {
      if (gi < ga.s && gj < ga.l) {  // parameter is l x s: element (gj, gi)
        const int64_t pidx = view_index(*md, gj, gi);
        if (ga.final_kind == 0) {
          const float w = load_as_f32(md->W, pidx, ga.param_dtype);
          store_from_f32(md->W, pidx, ga.param_dtype, fmaf(md->decay, w, -md->upd_scale * v));
        } else {
          store_from_f32(md->out, pidx, ga.param_dtype, v);
        }
      }
    } else {
      *reinterpret_cast<T*>(ga.CT + mat * ga.ct_mat + static_cast<int64_t>(gj) * ga.ldct + gi * static_cast<int>(sizeof(T))) = from_f32<T>(v);
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 C = P Q^T with a 256 x 256 output tile per workgroup (M and N
// multiples of 256).  512 threads = 8 wavefronts in a 2 x 4 grid, each owning
// a 128 x 64 sub-tile = 4 x 2 blocks of v_mfma_f32_32x32x16_bf16, so every
// operand fragment read from LDS feeds two or four MFMAs.
//
// K is staged 64 elements (128 bytes per row) at a time with direct
// global-to-LDS loads (global_load_lds_dwordx4: lane i of a wavefront writes
// bytes [16 i, 16 i + 16) after the wave-uniform LDS base), double-buffered.
// A wavefront instruction fills 8 consecutive tile rows; lane i fetches the
// 16-byte k-chunk (i % 8) ^ ((row >> 1) % 8) of its row, so LDS row r holds
// chunk c at position c ^ ((r >> 1) % 8).  A fragment read (32 rows, one
// chunk) then spreads over all 64 banks.
//
// The launch is persistent (one workgroup per CU).  Workgroup b runs on XCD
// b % 8; every round, the workgroups of one XCD take one compact block of the
// tile order (bands 8 tile-rows high), so they share operand panels in that
// XCD's L2.
//
// The epilogue works on the accumulator registers directly: lane l holds
// rows 8*(r/4) + 4*(l/32) + (r%4) of column l%32 in register r of a block, so
// 4 consecutive registers are 4 consecutive elements of a row of the
// transposed tile; a 4-lane transpose (DPP) gives the direct orientation.
// ---------------------------------------------------------------------------
// Compile-time loop: f(std::integral_constant<int, 0>) ... f(<N-1>), so array
// indices inside f are constants whatever the unroller decides.
template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}
template <int V>
using I_ = std::integral_constant<int, V>;

// Lane exchange inside each group of 4 lanes by DPP quad permutation: a VALU
// operand modifier, no LDS traffic.
constexpr int kQuadXor1 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;  // quad_perm [2,3,0,1]
template <int CTRL>
__device__ __forceinline__ uint32_t quad_swap(uint32_t x) {
  return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), CTRL, 0xF, 0xF, true));
}

// Lanes 4p..4p+3 each hold x[0..3] = M[t][0..3] (t = lane % 4); afterwards
// lane t holds M[0..3][t].  Two butterfly stages over lane bits 0 and 1.
// Every lane of the quad must be active.
__device__ __forceinline__ void quad_transpose(float x[4]) {
  const int t = threadIdx.x & 3;
  float y[4], n[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) y[k] = __uint_as_float(quad_swap<kQuadXor1>(__float_as_uint(x[k])));
#pragma unroll
  for (int r = 0; r < 4; ++r) n[r] = ((r ^ t) & 1) ? y[r ^ 1] : x[r];
#pragma unroll
  for (int k = 0; k < 4; ++k) y[k] = __uint_as_float(quad_swap<kQuadXor2>(__float_as_uint(n[k])));
#pragma unroll
  for (int r = 0; r < 4; ++r) x[r] = ((r ^ t) & 2) ? y[r ^ 2] : n[r];
}

// The same 4 x 4 transpose on packed bfloat16: d.x = M[t][0] | M[t][1] << 16,
// d.y = M[t][2] | M[t][3] << 16 becomes d.x = M[0][t] | M[1][t] << 16,
// d.y = M[2][t] | M[3][t] << 16.  Stage 1 swaps the off-diagonal 2 x 2
// blocks (whole dwords, lanes t ^ 2); stage 2 transposes inside each block
// (16-bit halves, lanes t ^ 1) with byte permutes.  8 VALU operations.
__device__ __forceinline__ uint2 quad_transpose_bf16(uint2 d) {
  const int t = threadIdx.x & 3;
  const bool hi_pair = (t & 2) != 0, odd = (t & 1) != 0;
  const uint32_t r1 = quad_swap<kQuadXor2>(hi_pair ? d.x : d.y);
  const uint32_t x1 = hi_pair ? r1 : d.x, y1 = hi_pair ? d.y : r1;
  // v_perm_b32(s0, s1, sel): selector bytes 0-3 pick bytes of s1, 4-7 of s0
  const uint32_t send = __builtin_amdgcn_perm(y1, x1, odd ? 0x05040100u : 0x07060302u);
  const uint32_t r2 = quad_swap<kQuadXor1>(send);
  return uint2{__builtin_amdgcn_perm(r2, x1, odd ? 0x03020504u : 0x05040100u),
               __builtin_amdgcn_perm(r2, y1, odd ? 0x03020706u : 0x07060100u)};
}

#ifndef MUON_NT
#define MUON_NT 1
#endif
// Epilogue outputs are written once and read by a later launch: streaming
// (non-temporal) stores keep them from displacing operand data in L2.
__device__ __forceinline__ void store_out(uint2* p, uint2 v) {
  if (MUON_NT) {
    __builtin_nontemporal_store(v.x, &p->x);
    __builtin_nontemporal_store(v.y, &p->y);
  } else {
    *p = v;
  }
}
__device__ __forceinline__ void store_out(u32x4_t* p, u32x4_t v) {
  if (MUON_NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}
__device__ __forceinline__ uint2 load_once(const uint2* p) {
  if (MUON_NT) return uint2{__builtin_nontemporal_load(&p->x), __builtin_nontemporal_load(&p->y)};
  return *p;
}

__device__ __forceinline__ uint2 pack_bf16x4(const float v[4]) {
  return uint2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
}
__device__ __forceinline__ void unpack_bf16x4(uint2 p, float v[4]) {
  v[0] = __uint_as_float(p.x << 16); v[1] = __uint_as_float(p.x & 0xffff0000u);
  v[2] = __uint_as_float(p.y << 16); v[3] = __uint_as_float(p.y & 0xffff0000u);
}

// Ragged-edge tail of apply4 (kept out of line: it is rare, and keeping the
// epilogue small lets the compiler hold every accumulator in registers).
template <int FK, int PDT>
__device__ __noinline__ void apply_tail(const MatDesc* md, int64_t idx, float o0, float o1, float o2,
                                        float o3, int n) {
  using PT = typename std::conditional<PDT == DT_BF16, uint16_t, float>::type;
  PT* dst = static_cast<PT*>(FK == 0 ? md->W : md->out);
  const float o[4] = {o0, o1, o2, o3};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if (q < n) {
      const float r = FK == 0 ? fmaf(md->decay, to_f32<PT>(dst[idx + q]), -md->upd_scale * o[q]) : o[q];
      dst[idx + q] = from_f32<PT>(r);
    }
  }
}

// W[idx .. idx+3] = decay*W - upd*o (FK = 0) or out[idx ..] = o (FK = 1), 4
// consecutive elements of dtype PDT: one vector access when `vec`, else
// element by element up to `n`.  The parameter is read and written with
// ordinary (cached) accesses, each load right before its store: measured
// faster than streaming accesses or loads hoisted ahead of the stores.
template <int FK, int PDT>
__device__ __forceinline__ void apply4(const MatDesc* md, int64_t idx, const float o[4], bool vec, int n) {
  using PT = typename std::conditional<PDT == DT_BF16, uint16_t, float>::type;
  PT* dst = static_cast<PT*>(FK == 0 ? md->W : md->out);
  const float decay = md->decay, upd = md->upd_scale;
  if (vec) {
    float w[4] = {0.f, 0.f, 0.f, 0.f}, r[4];
    if constexpr (PDT == DT_BF16) {
      uint2* p = reinterpret_cast<uint2*>(dst + idx);
      if (FK == 0) unpack_bf16x4(*p, w);
#pragma unroll
      for (int q = 0; q < 4; ++q) r[q] = FK == 0 ? fmaf(decay, w[q], -upd * o[q]) : o[q];
      *p = pack_bf16x4(r);
    } else {
      float4* p = reinterpret_cast<float4*>(dst + idx);
      if (FK == 0) {
        const float4 raw = *p;
        w[0] = raw.x; w[1] = raw.y; w[2] = raw.z; w[3] = raw.w;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) r[q] = FK == 0 ? fmaf(decay, w[q], -upd * o[q]) : o[q];
      *p = make_float4(r[0], r[1], r[2], r[3]);
    }
    return;
  }
  apply_tail<FK, PDT>(md, idx, o[0], o[1], o[2], o[3], n);
}

// Byte offset of an LDS object.
__device__ __forceinline__ uint32_t lds_offset(const char* p) {
  return static_cast<uint32_t>(
      reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) char*)(p)));
}

// Direct global -> LDS load (global_load_lds_dwordx4): lane i writes the 16
// bytes at base + off (base wave-uniform, off a 32-bit lane offset) to LDS
// bytes [lds + 16 i, lds + 16 i + 16); `lds` is wave-uniform.  Issued as
// inline assembly so that the compiler keeps no record of it: the kernel
// waits for these loads explicitly (vmcnt) before the barrier that publishes
// a slab, and the transposing LDS reads of the other stage must not wait for
// them.  M0 is set inside the statement.
__device__ __forceinline__ void load_lds16(const char* base, uint32_t off, uint32_t lds) {
  // (readfirstlane returns int: widen each half as unsigned, never by sign)
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b >> 32)));
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b & 0xffffffffu)));
  const uint64_t bs = (static_cast<uint64_t>(hi) << 32) | static_cast<uint64_t>(lo);
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(off), "s"(bs), "s"(__builtin_amdgcn_readfirstlane(lds)) : "memory");
}

// 8 bytes per lane from LDS through the transposing read (ds_read_b64_tr_b16).
__device__ __forceinline__ uint2 tr_read_b64(const char* p) {
  typedef short v4i16 __attribute__((ext_vector_type(4)));
  const v4i16 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4i16*)(const_cast<char*>(p)));
  return __builtin_bit_cast(uint2, v);
}

// Tile configuration of the direct-to-LDS MFMA kernel: output tile BM x BN,
// a WM x WN grid of wavefronts (each BM/WM x BN/WN), SLAB bytes of every
// tile row staged per LDS stage, NS stages, WPE wavefronts per SIMD.
template <int BM_, int BN_, int WM_, int WN_, int SLAB_, int NS_, int WPE_>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, SLAB = SLAB_, NS = NS_, WPE = WPE_;
  static constexpr int NW = WM * WN;
  static constexpr int LDS = NS * (BM + BN) * SLAB;
  static_assert(LDS <= 160 * 1024, "LDS budget");
};
// 256 x 256, 8 wavefronts, one workgroup per CU (symmetric products).
#ifndef MUON_SQ_SLAB
#define MUON_SQ_SLAB 128
#define MUON_SQ_STAGES 2
#endif
using CfgSquare = TileCfg<256, 256, 2, 4, MUON_SQ_SLAB, MUON_SQ_STAGES, 2>;

// Tile `logical` of the launch: matrix-major; inside a matrix, banded
// (GS / GM tile-rows per band, column by column inside a band).
__device__ __forceinline__ void tile_from_logical(const GemmArgs& ga, int logical, int& mat, int& bm,
                                                  int& bn) {
  mat = logical / ga.tiles_per_mat;
  int t = logical - mat * ga.tiles_per_mat;
  if (ga.syrk) {
    // upper-triangle tiles (bm <= bn) in bands of GS tile-rows, column by
    // column inside a band, so concurrent tiles share row and column panels
#ifndef MUON_GS
#define MUON_GS 8
#endif
    constexpr int GS = MUON_GS;
    const int T = ga.tiles_m;
    int b0 = 0;
    for (;;) {
      const int rows = min(GS, T - b0);
      const int size = rows * (rows + 1) / 2 + (T - b0 - rows) * rows;
      if (t < size) break;
      t -= size;
      b0 += GS;
    }
    const int rows = min(GS, T - b0);
    int c = 0;
    while (t >= min(rows, c + 1)) { t -= min(rows, c + 1); ++c; }
    bn = b0 + c;
    bm = b0 + t;
  } else {
#ifndef MUON_GM
#define MUON_GM 8
#endif
    constexpr int GM = MUON_GM;
    const int band = t / (GM * ga.tiles_n);
    const int within = t - band * GM * ga.tiles_n;
    const int rows = min(GM, ga.tiles_m - band * GM);
    bm = band * GM + within % rows;
    bn = within / rows;
  }
}

template <int EPI, class Cfg>
__device__ __forceinline__ void gemm_tile_body(const GemmArgs& ga, char* smem, int mat, int bm, int bn) {
  constexpr int BM = Cfg::BM, BN = Cfg::BN, WM = Cfg::WM, WN = Cfg::WN, NW = Cfg::NW;
  constexpr int SLAB = Cfg::SLAB, NS = Cfg::NS;
  constexpr int BI = BM / WM / 32;            // 32x32 blocks per wave, rows
  constexpr int BJ = BN / WN / 32;            // and columns
  constexpr int CPR = SLAB / 16;              // 16-byte chunks per staged row
  constexpr int SH = CPR == 8 ? 1 : 2;        // swizzle key: (row >> SH) & (CPR - 1)
  constexpr int RPI = 1024 / SLAB;            // rows one wave load instruction fills
  constexpr int PR = BM / NW, QR = BN / NW;   // operand rows each wave loads
  constexpr int NLP = PR / RPI, NLQ = QR / RPI;
  static_assert(NLP * RPI == PR && NLQ * RPI == QR, "load split");
  constexpr int GPS = SLAB / 32;              // 16-k MFMA groups per slab
  constexpr int OPQ = BM * SLAB;              // Q slab offset in a stage
  constexpr int STAGE = (BM + BN) * SLAB;
  constexpr bool FINAL = EPI >= EPI_FINAL_W_BF16;
  constexpr int FK = (EPI == EPI_FINAL_O_BF16 || EPI == EPI_FINAL_O_F32) ? 1 : 0;
  constexpr int PDT = (EPI == EPI_FINAL_W_F32 || EPI == EPI_FINAL_O_F32) ? DT_F32 : DT_BF16;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  static_assert(SLAB == 128 && NS == 2 && GPS == 4 && BM * 2 == 512 && BN * 2 == 512 && RPI == 8,
                "slab geometry: 64 k of 256 rows, or 64 k-rows of 256 columns");

  // ---- operand slabs ---------------------------------------------------------
  // A slab holds 64 consecutive k of the tile's 256 rows of P (and of Q), in
  // one of two geometries:
  //  - direct: 256 rows of 128 bytes (k contiguous), for an operand stored
  //    row-major over k;
  //  - transposed: 64 rows k of 512 bytes (the tile's rows contiguous), for
  //    an operand stored K x rows, read back with ds_read_b64_tr_b16.
  // Mode 0 reads every slab direct; mode 2 (Q only) every slab transposed:
  // the update products read X itself as their second operand.  Mode 1 is
  // the symmetric matrices A and B stored as their upper-triangle 256 x 256
  // tiles only: rows of tile-row b below the diagonal block (k < 256 b) are
  // columns of the stored tile (k-block, b), read transposed.
  const int nk = ga.k_slabs;
  const int p_tr_end = ga.p_mode == 1 ? bm * (BM / 64) : 0;   // slabs [0, p_tr_end) transposed
  const int q_tr_end = ga.q_mode == 2 ? nk : (ga.q_mode == 1 ? bn * (BN / 64) : 0);
  constexpr bool QTR = EPI == EPI_UPDATE || FINAL;           // update products: Q always transposed
  constexpr bool CAN_PT = EPI != EPI_GRAM, CAN_QT = EPI != EPI_GRAM, CAN_QD = !QTR;
  const char* const Pm = ga.P + mat * ga.p_mat;
  const char* const Qm = ga.Q + mat * ga.q_mat;
  const char* const Pd = Pm + static_cast<int64_t>(bm) * BM * ga.ldp;   // + ks * SLAB
  const char* const Qd = Qm + static_cast<int64_t>(bn) * BN * ga.ldq;
  const char* const Pt = Pm + bm * BM * 2;                               // + ks * 64 * ld
  const char* const Qt = Qm + bn * BN * 2;

  // Loads: a wave instruction fills 1 KB of the stage (8 direct rows or 2
  // transposed rows); lane l writes 16 bytes at 16 l and fetches the chunk
  // that belongs there.  Direct: LDS row r holds k-chunk c at position
  // c ^ ((r >> 1) % 8), which spreads the 32 rows of a fragment read over all
  // 64 banks.  Transposed: row k holds 16-byte chunk c at position
  // c ^ 4*(k % 4).  Per-lane offsets are 32-bit, added to a wave-uniform base.
  uint32_t pdo[NLP], pto[NLP], qdo[NLQ], qto[NLQ];
#pragma unroll
  for (int i = 0; i < NLP; ++i) {
    const int r = wave * PR + RPI * i + lane / CPR;
    pdo[i] = static_cast<uint32_t>(r * ga.ldp + ((lane % CPR) ^ ((r >> SH) & (CPR - 1))) * 16);
    const int t = wave * (2 * NLP) + 2 * i + lane / 32;
    pto[i] = static_cast<uint32_t>(t * ga.ldp + ((lane % 32) ^ ((t & 3) << 2)) * 16);
  }
#pragma unroll
  for (int i = 0; i < NLQ; ++i) {
    const int r = wave * QR + RPI * i + lane / CPR;
    qdo[i] = static_cast<uint32_t>(r * ga.ldq + ((lane % CPR) ^ ((r >> SH) & (CPR - 1))) * 16);
    const int t = wave * (2 * NLQ) + 2 * i + lane / 32;
    qto[i] = static_cast<uint32_t>(t * ga.ldq + ((lane % 32) ^ ((t & 3) << 2)) * 16);
  }
  const uint32_t lds0 = lds_offset(smem);
  // The loads of slab ks, one operand at a time: P's NLP instructions or Q's
  // NLQ, into the slab's stage.
  auto issue_op = [&](auto qc, int ks) __attribute__((always_inline)) {
    const uint32_t base = lds0 + (ks & 1) * STAGE;
    if constexpr (!decltype(qc)::value) {
      if (CAN_PT && ks < p_tr_end) {
        const char* b = Pt + static_cast<int64_t>(ks) * 64 * ga.ldp;
#pragma unroll
        for (int i = 0; i < NLP; ++i) load_lds16(b, pto[i], base + (wave * PR + RPI * i) * SLAB);
      } else {
        const char* b = Pd + ks * SLAB;
#pragma unroll
        for (int i = 0; i < NLP; ++i) load_lds16(b, pdo[i], base + (wave * PR + RPI * i) * SLAB);
      }
    } else {
      if (CAN_QT && (!CAN_QD || ks < q_tr_end)) {
        const char* b = Qt + static_cast<int64_t>(ks) * 64 * ga.ldq;
#pragma unroll
        for (int i = 0; i < NLQ; ++i) load_lds16(b, qto[i], base + OPQ + (wave * QR + RPI * i) * SLAB);
      } else {
        const char* b = Qd + ks * SLAB;
#pragma unroll
        for (int i = 0; i < NLQ; ++i) load_lds16(b, qdo[i], base + OPQ + (wave * QR + RPI * i) * SLAB);
      }
    }
  };
  auto issue = [&](int ks) __attribute__((always_inline)) {
    issue_op(std::false_type{}, ks);
    issue_op(std::true_type{}, ks);
  };

  f32x16_t acc[BI][BJ];
#pragma unroll
  for (int i = 0; i < BI; ++i)
#pragma unroll
    for (int j = 0; j < BJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Fragments.  Direct: row (.. + lane % 32), k-chunk 2*grp + lane / 32 at its
  // swizzled position, one ds_read_b128.  Transposed: ds_read_b64_tr_b16
  // hands lane t of each 16-lane group G, as its r-th element, element t % 4
  // of the 8 bytes addressed by lane 4r + t / 4 of the group.  Lane L of
  // group G therefore addresses row 16*grp + 8*(G/2) + 4*h + L/4, columns
  // c0 + 16*(G%2) + 4*(L%4) .. +3, and two reads (h = 0, 1) give the 8
  // consecutive k of column c0 + lane % 32 that the MFMA takes.  The 4 rows k
  // of one read differ in k % 4, so the swizzle spreads them over all banks.
  const int frow = lane & 31, fsel = lane >> 5, fsw = (frow >> SH) & (CPR - 1);
  const int a_off = (wm * (BM / WM) + frow) * SLAB;
  const int b_off = OPQ + (wn * (BN / WN) + frow) * SLAB;
  auto tr_off = [&](int c0) {
    const int G = lane >> 4, L = lane & 15;
    const int row = 8 * (G >> 1) + (L >> 2);
    const int cb = 2 * c0 + 32 * (G & 1) + 8 * (L & 3);
    return row * 512 + (cb ^ ((L >> 2) << 6));
  };
  int tpo[BI], tqo[BJ];
#pragma unroll
  for (int i = 0; i < BI; ++i) tpo[i] = tr_off(wm * (BM / WM) + i * 32);
#pragma unroll
  for (int j = 0; j < BJ; ++j) tqo[j] = OPQ + tr_off(wn * (BN / WN) + j * 32);

  // ---- the a*X (or A) term, taken from the operand slabs ----------------------
  // The tile that the epilogue combines with the product passes through LDS
  // as part of an operand, so it is added to the accumulators there instead
  // of being read from memory again:
  //  - update products: rows bm*256 + [0, 256) of X are the Q slabs
  //    4 bm .. 4 bm + 3 (transposed geometry); the wave's 128 rows are slabs
  //    4 bm + 2 wm + h, h = 0, 1, holding its row blocks 2h and 2h + 1;
  //  - polynomial: A[bm, bn] is the P slabs 4 bn .. 4 bn + 3 (direct, as
  //    bn >= bm); the wave's 64 columns are slab 4 bn + wn.
  // One transposing read gives a lane the 4 consecutive rows of one column
  // that 4 accumulator registers hold: lane 4e + q of 16-lane group G
  // addresses row 4(G/2) + e, columns 16(G%2) + 4q .. +3 of the block's
  // register group, and lane t receives column 16(G%2) + t, rows 0..3.
  // The polynomial adds alpha = b/c times A and scales by beta = c at the
  // end; with c = 0 the launch keeps the epilogue path (e_loop = 0).
  constexpr bool EUPD = QTR;
  constexpr int EPS = (BN / WN) / 64;           // P slabs holding a wave's columns of A
  static_assert(EPS == 1 || EPS == 2, "A term: one or two slabs per wave");
  constexpr int EJ = BJ / EPS;                  // 32-column blocks per such slab
  const bool epoly = EPI == EPI_POLY && ga.e_loop != 0;
  int e_ks0 = -1, e_ks1 = -1;
  if (EUPD) {
    e_ks0 = bm * (BM / 64) + 2 * wm;
    e_ks1 = e_ks0 + 1;
  } else if (epoly) {
    // the wave's BN / WN columns are EPS slabs of 64 k
    e_ks0 = bn * (BN / 64) + wn * EPS;
    if (EPS > 1) e_ks1 = e_ks0 + 1;
  }
  int eo[BJ][2];
  {
    const int G = lane >> 4, L = lane & 15;
#pragma unroll
    for (int j = 0; j < BJ; ++j)
#pragma unroll
      for (int gp = 0; gp < 2; ++gp) {
        if (EUPD)  // Q slab: row k holds chunk c at c ^ 4(k % 4)
          eo[j][gp] = OPQ + (4 * (G >> 1) + (L >> 2)) * 512 +
                      ((2 * (wn * (BN / WN) + 32 * j) + 32 * (G & 1) + 8 * (L & 3)) ^ ((L >> 2) << 6));
        else       // P slab: row r holds chunk c at c ^ ((r >> 1) % 8)
          eo[j][gp] = (wm * (BM / WM) + 4 * (G >> 1) + (L >> 2)) * SLAB +
                      (((4 * (j % EJ) + 2 * (G & 1) + ((L >> 1) & 1)) ^ (4 * gp + 2 * (G >> 1) + (L >> 3))) << 4) +
                      8 * (L & 1);
      }
  }
  // Rows [i0, i0 + ni) and 32-column blocks [j0, j0 + nj) of the wave's
  // accumulators take the term from the slab at sp.
  auto add_e = [&](const char* sp, auto i0c, auto nic, auto j0c, auto njc) __attribute__((always_inline)) {
    constexpr int i0 = decltype(i0c)::value, ni = decltype(nic)::value;
    constexpr int j0 = decltype(j0c)::value, nj = decltype(njc)::value;
    static_for<ni>([&](auto II) {
      constexpr int i = i0 + decltype(II)::value;
      uint2 ev[nj][4];
      static_for<nj>([&](auto J) {
        static_for<4>([&](auto Gc) {
          constexpr int jj = decltype(J)::value, j = j0 + jj, g = decltype(Gc)::value;
          ev[jj][g] = EUPD ? tr_read_b64(sp + eo[j][0] + (32 * (i & 1) + 8 * g) * 512)
                           : tr_read_b64(sp + eo[j][g & 1] + (32 * i + 8 * g) * SLAB);
        });
      });
      static_for<nj>([&](auto J) {
        static_for<4>([&](auto Gc) {
          constexpr int jj = decltype(J)::value, j = j0 + jj, g = decltype(Gc)::value;
          float e[4];
          unpack_bf16x4(ev[jj][g], e);
          f32x16_t& c = acc[i][j];
          c[4 * g + 0] = fmaf(ga.alpha, e[0], c[4 * g + 0]);
          c[4 * g + 1] = fmaf(ga.alpha, e[1], c[4 * g + 1]);
          c[4 * g + 2] = fmaf(ga.alpha, e[2], c[4 * g + 2]);
          c[4 * g + 3] = fmaf(ga.alpha, e[3], c[4 * g + 3]);
        });
      });
    });
  };

  // Software pipeline: the fragments of group g+1 are read into the other
  // register set while group g's MFMAs issue, one LDS read between
  // consecutive MFMAs; the slab barrier sits before the last group's MFMAs.
  u32x4_t fa[2][BI], fb[2][BJ];
  auto rd = [&](auto ptc, auto qtc, const char* sp, auto grpc, auto setc) __attribute__((always_inline)) {
    constexpr bool PT = decltype(ptc)::value, QT = decltype(qtc)::value;
    constexpr int grp = decltype(grpc)::value, set = decltype(setc)::value;
    const int pos = ((2 * grp + fsel) ^ fsw) * 16;
#pragma unroll
    for (int i = 0; i < BI; ++i) {
      if (PT) {
        const char* q = sp + tpo[i] + grp * 16 * 512;
        const uint2 lo = tr_read_b64(q), hi = tr_read_b64(q + 4 * 512);
        fa[set][i] = u32x4_t{lo.x, lo.y, hi.x, hi.y};
      } else {
        fa[set][i] = *reinterpret_cast<const u32x4_t*>(sp + a_off + i * 32 * SLAB + pos);
      }
    }
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
      if (QT) {
        const char* q = sp + tqo[j] + grp * 16 * 512;
        const uint2 lo = tr_read_b64(q), hi = tr_read_b64(q + 4 * 512);
        fb[set][j] = u32x4_t{lo.x, lo.y, hi.x, hi.y};
      } else {
        fb[set][j] = *reinterpret_cast<const u32x4_t*>(sp + b_off + j * 32 * SLAB + pos);
      }
    }
  };
  auto mm = [&](auto setc) __attribute__((always_inline)) {
    constexpr int set = decltype(setc)::value;
    static_for<BI>([&](auto I) {
      static_for<BJ>([&](auto J) { Mma<uint16_t>::run(fa[set][I.value], fb[set][J.value], acc[I.value][J.value]); });
    });
  };
  auto interleave = [&](auto ptc, auto qtc) __attribute__((always_inline)) {
    constexpr int NRD = (decltype(ptc)::value ? 2 : 1) * BI + (decltype(qtc)::value ? 2 : 1) * BJ;
    constexpr int NPAIR = NRD < BI * BJ ? NRD : BI * BJ;
#pragma unroll
    for (int i = 0; i < NPAIR; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
    }
    if constexpr (BI * BJ > NPAIR) __builtin_amdgcn_sched_group_barrier(0x008, BI * BJ - NPAIR, 0);
    if constexpr (NRD > NPAIR) __builtin_amdgcn_sched_group_barrier(0x100, NRD - NPAIR, 0);
  };
  // One slab in mode (PT, QT); group 0's fragments are already in set 0.
  // With NEXT, the fragments of the next slab's group 0 (same mode) are read
  // while the last group's MFMAs issue; without, the last group runs alone
  // (the slab before a change of mode, and the last one).
  // When a slab's loads are issued, one operand at a time, so that the
  // workgroups of an XCD do not ask for a whole slab at once:
  //  - Gram product (EARLY): Q's right after the barrier that frees the
  //    stage, P's at the top of the next slab (the slab of lead that was
  //    measured faster for its long K);
  //  - the other products: Q's at the top of the slab before, P's after
  //    that slab's first MFMA group (3/4 and 1/2 of a slab ahead).
  // Splitting the burst by operand measured 2-3% faster on the step than
  // issuing a slab at once; splitting each operand in halves, or P later,
  // measured slower.
  constexpr bool EARLY = EPI == EPI_GRAM;
  auto slab = [&](auto ptc, auto qtc, auto nextc, auto ec, int ks) __attribute__((always_inline)) {
    const char* sp = smem + (ks & 1) * STAGE;
    if (ks + 1 < nk) {
      if (!EARLY) issue_op(std::true_type{}, ks + 1);
      else if (ks >= 1) issue_op(std::false_type{}, ks + 1);  // slab 1 went out whole with slab 0
    }
    if constexpr (decltype(ec)::value) {
      if (ks == e_ks0 || ks == e_ks1) {  // wave-uniform; at most twice a tile
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (EUPD) {
          if (ks == e_ks0) add_e(sp, I_<0>{}, I_<2>{}, I_<0>{}, I_<BJ>{});
          else add_e(sp, I_<2>{}, I_<2>{}, I_<0>{}, I_<BJ>{});
        } else if constexpr (EPS == 1) {
          add_e(sp, I_<0>{}, I_<BI>{}, I_<0>{}, I_<BJ>{});
        } else {
          if (ks == e_ks0) add_e(sp, I_<0>{}, I_<BI>{}, I_<0>{}, I_<EJ>{});
          else add_e(sp, I_<0>{}, I_<BI>{}, I_<EJ>{}, I_<EJ>{});
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    rd(ptc, qtc, sp, I_<1>{}, I_<1>{}); mm(I_<0>{}); interleave(ptc, qtc);
    __builtin_amdgcn_sched_barrier(0);
    if (!EARLY && ks + 1 < nk) issue_op(std::false_type{}, ks + 1);
    __builtin_amdgcn_sched_barrier(0);
    rd(ptc, qtc, sp, I_<2>{}, I_<0>{}); mm(I_<1>{}); interleave(ptc, qtc);
    __builtin_amdgcn_sched_barrier(0);
    rd(ptc, qtc, sp, I_<3>{}, I_<1>{}); mm(I_<0>{}); interleave(ptc, qtc);
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // slab ks + 1 has landed
    __syncthreads();
    // every wave is done with slab ks: its stage can take slab ks + 2
    if (EARLY && ks + 2 < nk) issue_op(std::true_type{}, ks + 2);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (decltype(nextc)::value) {
      rd(ptc, qtc, smem + ((ks + 1) & 1) * STAGE, I_<0>{}, I_<0>{});
      mm(I_<1>{}); interleave(ptc, qtc);
    } else {
      mm(I_<1>{});
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // Slabs [a, b) in one mode.  Each run starts from a published slab and
  // ends with the next one published, so runs chain without carrying
  // fragments across a change of mode (which happens at most twice a tile).
  // With ec, the run may hold the slabs that carry the a*X (or A) term.
  auto run = [&](auto ptc, auto qtc, auto ec, int a, int b) __attribute__((always_inline)) {
    if (a >= b) return;
    rd(ptc, qtc, smem + (a & 1) * STAGE, I_<0>{}, I_<0>{});
    for (int ks = a; ks < b - 1; ++ks) slab(ptc, qtc, std::true_type{}, ec, ks);
    slab(ptc, qtc, std::false_type{}, ec, b - 1);
  };
  using T_ = std::true_type;
  using F_ = std::false_type;
  issue(0);
  if (EARLY && nk > 1) {
    issue(1);
    // slab 0 has landed, slab 1 (NLP + NLQ loads) may not
    asm volatile("s_waitcnt vmcnt(%0)" :: "n"(NLP + NLQ) : "memory");
  } else {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
  __syncthreads();
  // Mode runs: P transposed for [0, p_tr_end), Q for [0, q_tr_end).  The
  // launches keep p_tr_end <= q_tr_end (GRAM none, POLY bm <= bn, update
  // products Q transposed throughout).
  // The term's slabs lie in the last run (k >= 256 bm for the update
  // products, k >= 256 bn for the polynomial).
  if constexpr (EPI == EPI_GRAM) {
    run(F_{}, F_{}, F_{}, 0, nk);
  } else if constexpr (QTR) {
    run(T_{}, T_{}, F_{}, 0, p_tr_end);
    run(F_{}, T_{}, T_{}, p_tr_end, nk);
  } else {
    run(T_{}, T_{}, F_{}, 0, p_tr_end);
    run(F_{}, T_{}, F_{}, p_tr_end, q_tr_end);
    run(F_{}, F_{}, T_{}, max(p_tr_end, q_tr_end), nk);
  }

  // ---- epilogue from registers ----------------------------------------------
  // Lane l holds, per 32x32 block and register group g, rows row0..row0+3 of
  // one column `col` (the natural layout: also 4 consecutive elements of row
  // `col` of the transposed tile).  A 4-lane transpose gives the direct
  // layout: lane t = l % 4 holds row row0+t, columns c0..c0+3, and 8 lanes
  // cover 64 contiguous bytes of a row.
  //  - The a*X (or A) term is already in the accumulators (added in the main
  //    loop), except for a polynomial launched with e_loop = 0, which reads
  //    it here, through the staging area or coalesced in the direct layout.
  //  - Outputs are rounded to bfloat16 once and leave through LDS as whole
  //    512-byte rows.  When the symmetric products must also write their
  //    mirrored tile (see below), that one is staged instead and the direct
  //    copy goes straight to memory.  X' needs no transposed copy, since the
  //    next update reads X through transposing LDS reads.
  //  - The last step's parameter update runs in the parameter's layout:
  //    direct when it is s x l, natural when it is l x s.
  //  - Every load of the a*X (or A) term is issued before the first store,
  //    so one memory latency is exposed instead of one per block.
  const bool diag = ga.syrk && bm == bn;
  const MatDesc* md = FINAL ? ga.desc + mat : nullptr;
  const bool tr = FINAL ? md->transposed != 0 : false;
  const bool v4 = FINAL ? md->vec4_ok != 0 : false;
  const int q4 = lane & 3;
  const int row_base = bm * BM + wm * (BM / WM) + 4 * fsel;
  const int col_base = bn * BN + wn * (BN / WN) + frow;
  char* const C = ga.C + mat * ga.c_mat;
  char* const CT = ga.CT + mat * ga.ct_mat;
  const char* const E = ga.E + mat * ga.e_mat;
  const char* const ET = ga.ET + mat * ga.et_mat;
  constexpr int TST = BM * 2 + 8;             // staged transposed row, bytes
  const bool stage_t = !QTR && ga.CT != nullptr;
  const bool stage_c = !FINAL && !stage_t;
  const bool e_epi = EPI == EPI_POLY && !epoly;  // the term is read in the epilogue
  // Natural staging (the output tile, no epilogue input): each lane's 4
  // consecutive rows of one column go to LDS as they are, 8 bytes at
  // column-major position (col, row) with a 520-byte column pitch, and the
  // copy-out reads whole rows back through transposing LDS reads.  No
  // register transposes; diagonal tiles of the symmetric products take
  // their lower triangle from the mirrored column at copy-out.
  const bool stage_n = stage_c && !e_epi;
  // The factor the accumulators leave with: c for a polynomial that added
  // (b/c) A in the main loop; on the first step, whose X holds u unscaled,
  // r^2 for the Gram product and r for the update products.
  float osc = 1.f;
  if (EPI == EPI_POLY) {
    osc = epoly ? ga.beta : 1.f;
  } else if (ga.xscale) {
    const float r = ga.xscale[mat];
    osc = EPI == EPI_GRAM ? r * r : r;
  }

  // Diagonal tiles of the symmetric products are written exactly symmetric:
  // the value computed for (row, col) with row <= col also goes to (col, row).
  // With a mirror (stage_t) this happens element by element in memory;
  // otherwise in the LDS staging area below.
  if (!FINAL && diag && stage_t) {
    static_for<BI>([&](auto I) {
      static_for<BJ>([&](auto J) {
        static_for<4>([&](auto G) {
          constexpr int i = decltype(I)::value, j = decltype(J)::value, g = decltype(G)::value;
          const int row0 = row_base + i * 32 + 8 * g;
          const int col = col_base + j * 32;
          float v[4];
          if (!e_epi) {
#pragma unroll
            for (int q = 0; q < 4; ++q) v[q] = osc * acc[i][j][4 * g + q];
          } else {
            float e[4];
            unpack_bf16x4(*reinterpret_cast<const uint2*>(ET + static_cast<int64_t>(col) * ga.ldet + row0 * 2), e);
#pragma unroll
            for (int q = 0; q < 4; ++q)
              v[q] = EPI == EPI_POLY ? fmaf(ga.alpha, e[q], ga.beta * acc[i][j][4 * g + q])
                                     : fmaf(ga.alpha, e[q], acc[i][j][4 * g + q]);
          }
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int row = row0 + q;
            if (row <= col) {
              const uint16_t h = f32_to_bf16(v[q]);
              *reinterpret_cast<uint16_t*>(C + static_cast<int64_t>(row) * ga.ldc + col * 2) = h;
              *reinterpret_cast<uint16_t*>(C + static_cast<int64_t>(col) * ga.ldc + row * 2) = h;
            }
          }
        });
      });
    });
    return;
  }

  // The symmetric products also write the mirrored tile, staged through LDS,
  // unless their consumers read the upper triangle only (CT null).  Without
  // a mirror, the output tile itself goes through LDS (stage_c): the a*X (or
  // A) tile is loaded into it as whole 512-byte rows by direct-to-LDS loads,
  // every lane combines its values in place, and the result leaves as whole
  // rows again, which measured faster than 64-byte row pieces to and from
  // the registers.  Staged rows are 512 bytes; row r holds 16-byte chunk c at
  // position c ^ 4*(r % 4), so the 8 rows x 64 bytes a lane instruction
  // touches spread over all banks.
  auto cpos = [](int r, int b) {  // staged byte position of tile row r, byte b
    return r * (BN * 2) + ((((b >> 4) ^ ((r & 3) << 2))) << 4) + (b & 15);
  };
  // The last step with a bfloat16 parameter whose 256 x 256 block lies fully
  // inside the matrix (and 16-byte rows): W goes through LDS the same way,
  // loaded and written back as whole 512-byte rows of its own layout.  Its
  // staged row r holds chunk c at c ^ key(r), key(r) = 4*(r % 4) + (r / 4) % 4,
  // which spreads both the direct accesses (8 rows x 64 bytes) and the
  // natural ones (32 rows x 16 bytes) over all banks.
  bool stage_w = false;
  if constexpr (FINAL && FK == 0 && PDT == DT_BF16)
    stage_w = v4 && md->cols % 8 == 0 && md->ld % 8 == 0 && md->rb >= md->rows &&
              md->ld * 2 < kTileMaxRowBytes && (bm + 1) * BM <= ga.s && (bn + 1) * BN <= ga.l;
  auto wpos = [](int r, int b) {
    const int key = ((r & 3) << 2) | ((r >> 2) & 3);
    return r * 512 + (((b >> 4) ^ key) << 4) + (b & 15);
  };
  const int wr0 = tr ? bn * BN : bm * BM, wc0 = tr ? bm * BM : bn * BN;  // W block origin
  // (every wave finished its operand-slab reads before the last slab's
  // barrier, so the staging area, which overlaps the slabs, is free)
  if (stage_w) {
    constexpr int KW = BM * BN * 2 / 1024 / NW;   // load instructions per wave
    static_assert(KW * NW * 1024 == BM * BN * 2, "W tile: whole instructions per wave");
    const char* wb = static_cast<const char*>(md->W) + (static_cast<int64_t>(wr0) * md->ld + wc0) * 2;
    const uint32_t ldw = static_cast<uint32_t>(md->ld) * 2;
    const uint32_t lds0 = lds_offset(smem);
#pragma unroll
    for (int k = 0; k < KW; ++k) {
      const int row = 2 * (wave * KW + k) + lane / 32;
      const int c = (lane % 32) ^ (((row & 3) << 2) | ((row >> 2) & 3));
      load_lds16(wb, static_cast<uint32_t>(row) * ldw + static_cast<uint32_t>(c * 16), lds0 + (wave * KW + k) * 1024);
    }
  }
  if (e_epi && stage_c) {
    // a wave instruction fills 2 staged rows (1 KB); lane l: row 2k + l/32,
    // position l % 32, which holds chunk (l % 32) ^ 4*(row % 4)
    constexpr int KE = BM * BN * 2 / 1024 / NW;   // load instructions per wave
    static_assert(KE * NW * 1024 == BM * BN * 2, "E tile: whole instructions per wave");
    const char* eb = E + static_cast<int64_t>(bm) * BM * ga.lde + bn * BN * 2;
    const uint32_t lds0 = lds_offset(smem);
#pragma unroll
    for (int k = 0; k < KE; ++k) {
      const int row = 2 * (wave * KE + k) + lane / 32;
      const int c = (lane % 32) ^ ((row & 3) << 2);
      load_lds16(eb, static_cast<uint32_t>(row * ga.lde + c * 16), lds0 + (wave * KE + k) * 1024);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }
  // (The loads and the per-block work sit in one lambda: inlined that way the
  // compiler keeps every value in registers; written at function scope it
  // spilled.)
  auto blocks = [&]() {
    uint2 ev[BI][BJ][4];
    static_for<BI>([&](auto I) {
      static_for<BJ>([&](auto J) {
        static_for<4>([&](auto G) {
          constexpr int i = decltype(I)::value, j = decltype(J)::value, g = decltype(G)::value;
          const int row0 = row_base + i * 32 + 8 * g;
          const int c0 = col_base + j * 32 - q4;
          if (e_epi && !stage_c)
            ev[i][j][g] = load_once(reinterpret_cast<const uint2*>(E + static_cast<int64_t>(row0 + q4) * ga.lde + c0 * 2));
          else if (e_epi && diag)  // the mirrored writes below reach other lanes' inputs
            ev[i][j][g] = *reinterpret_cast<const uint2*>(smem + cpos(row0 + q4 - bm * BM, (c0 - bn * BN) * 2));
        });
      });
    });
    if (e_epi && stage_c && diag) __syncthreads();
    if (stage_w) {  // the W block has landed in LDS
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
    }
    const float decay = FINAL ? md->decay : 0.f, upd = FINAL ? md->upd_scale : 0.f;
    auto w_update = [&](char* p, const float o[4]) {  // 4 staged W values, in place
      float w[4], r[4];
      unpack_bf16x4(*reinterpret_cast<const uint2*>(p), w);
#pragma unroll
      for (int q = 0; q < 4; ++q) r[q] = fmaf(decay, w[q], -upd * o[q]);
      *reinterpret_cast<uint2*>(p) = pack_bf16x4(r);
    };
    static_for<BI>([&](auto I) {
      static_for<BJ>([&](auto J) {
        static_for<4>([&](auto G) {
          constexpr int i = decltype(I)::value, j = decltype(J)::value, g = decltype(G)::value;
          const int row0 = row_base + i * 32 + 8 * g;  // rows row0 .. row0 + 3
          const int col = col_base + j * 32;
          const int c0 = col - q4;                     // direct layout: columns c0 .. c0 + 3
          float v[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) v[q] = acc[i][j][4 * g + q] * (e_epi ? 1.f : osc);
          if (!FINAL || tr) {  // natural layout
            if (e_epi) {
              float e[4];
              const uint2 ed = (stage_c && !diag) ? *reinterpret_cast<const uint2*>(smem + cpos(row0 + q4 - bm * BM, (c0 - bn * BN) * 2))
                                                  : ev[i][j][g];
              unpack_bf16x4(quad_transpose_bf16(ed), e);
#pragma unroll
              for (int q = 0; q < 4; ++q) v[q] = fmaf(ga.alpha, e[q], ga.beta * v[q]);
            }
            if (stage_n) {
              *reinterpret_cast<uint2*>(smem + (col - bn * BN) * TST + (row0 - bm * BM) * 2) = pack_bf16x4(v);
            } else if (!FINAL && diag) {  // stage_c: (row, col) and (col, row) for row <= col
              const int cl = col - bn * BN;
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const int rl = row0 + q - bm * BM;
                if (rl <= cl) {
                  const uint16_t h = f32_to_bf16(v[q]);
                  *reinterpret_cast<uint16_t*>(smem + cpos(rl, cl * 2)) = h;
                  *reinterpret_cast<uint16_t*>(smem + cpos(cl, rl * 2)) = h;
                }
              }
            } else if (!FINAL) {
              const uint2 p = pack_bf16x4(v);
              const uint2 d = quad_transpose_bf16(p);  // row row0 + q4, columns c0 .. c0 + 3
              if (stage_c) {
                *reinterpret_cast<uint2*>(smem + cpos(row0 + q4 - bm * BM, (c0 - bn * BN) * 2)) = d;
              } else {
                *reinterpret_cast<uint2*>(smem + (col - bn * BN) * TST + (row0 - bm * BM) * 2) = p;
                store_out(reinterpret_cast<uint2*>(C + static_cast<int64_t>(row0 + q4) * ga.ldc + c0 * 2), d);
              }
            } else if (stage_w) {      // parameter is l x s: elements (col, row0 .. row0 + 3)
              w_update(smem + wpos(col - wr0, (row0 - wc0) * 2), v);
            } else if (col < ga.l) {
              const int n = min(4, ga.s - row0);
              if (n > 0)
                apply4<FK, PDT>(md, view_index(*md, col, row0), v, v4 && n == 4, n);
            }
          } else {             // parameter is s x l: elements (row0 + q4, c0 .. c0 + 3)
            quad_transpose(v);
            const int row = row0 + q4;
            if (stage_w) {
              w_update(smem + wpos(row - wr0, (c0 - wc0) * 2), v);
            } else if (row < ga.s) {
              const int n = min(4, ga.l - c0);
              if (n > 0)
                apply4<FK, PDT>(md, view_index(*md, row, c0), v, v4 && n == 4, n);
            }
          }
        });
      });
    });
  };
  blocks();
  if (stage_w) {
    __syncthreads();
    // updated W rows (512 bytes each) -> W, 16 bytes a thread
    for (int idx = threadIdx.x; idx < BM * 32; idx += 64 * NW) {
      const int r = idx >> 5, ch = idx & 31;
      *reinterpret_cast<u32x4_t*>(static_cast<char*>(md->W) + (static_cast<int64_t>(wr0 + r) * md->ld + wc0) * 2 +
                                  ch * 16) = *reinterpret_cast<const u32x4_t*>(smem + wpos(r, ch * 16));
    }
    __syncthreads();  // the next tile's loads overwrite the staging area
  }
  if (stage_n) {
    __syncthreads();
    // Copy-out: a wave instruction writes 4 rows x 256 bytes.  In each
    // 16-lane group G, lane t (r = t / 4, q = t % 4) addresses the 8 bytes
    // (rows R .. R + 3) of column C0 + 8 q + r, then of column C0 + 8 q + 4 + r;
    // ds_read_b64_tr_b16 hands lane t row R + t % 4, columns C0 + 8 (t / 4)
    // .. + 3 and + 4 .. + 7: 16 consecutive bytes of one row.
    const int G = lane >> 4, t = lane & 15;
    const int ra = ((t & 3) * 8 + (t >> 2)) * TST;     // column offset of this lane's first address
    const int rrow = t & 3, rcol = 8 * (t >> 2);       // what it receives
    constexpr int KC = BM * BN * 2 / 1024 / NW;   // store instructions per wave
    static_assert(KC * NW * 1024 == BM * BN * 2, "copy-out: whole instructions per wave");
    auto out_row = [&](int it, auto diagc) __attribute__((always_inline)) {
      const int task = it * NW + wave;                 // 4 rows x 128 columns
      const int R = 4 * (task >> 1), C0 = 128 * (task & 1) + 32 * G;
      const char* a = smem + C0 * TST + ra + 2 * R;
      const uint2 lo = tr_read_b64(a), hi = tr_read_b64(a + 4 * TST);
      u32x4_t v{lo.x, lo.y, hi.x, hi.y};
      const int row = R + rrow, c = C0 + rcol;
      if (decltype(diagc)::value && c < row) {
        // columns c .. c + 7 below the diagonal hold (col, row): row `row`
        // of the staged column-major tile, i.e. column `row`, rows c ..
        const char* m = smem + row * TST + 2 * c;
        const uint2 l0 = *reinterpret_cast<const uint2*>(m), l1 = *reinterpret_cast<const uint2*>(m + 8);
        const u32x4_t low{l0.x, l0.y, l1.x, l1.y};
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          const int c2 = c + 2 * d;                    // elements c2 (low half) and c2 + 1
          v[d] = c2 + 1 < row ? low[d] : (c2 < row ? ((low[d] & 0xffffu) | (v[d] & 0xffff0000u)) : v[d]);
        }
      }
      store_out(reinterpret_cast<u32x4_t*>(C + static_cast<int64_t>(bm * BM + row) * ga.ldc + (bn * BN + c) * 2), v);
    };
    if (diag) {
      for (int it = 0; it < KC; ++it) out_row(it, std::true_type{});
    } else {
#pragma unroll
      for (int it = 0; it < KC; ++it) out_row(it, std::false_type{});
    }
    __syncthreads();  // the next tile's loads overwrite the staging area
  } else if (stage_c) {
    __syncthreads();
    // output tile rows (BN bf16 = 512 bytes each) -> C, 16 bytes a thread
    constexpr int CH = BN * 2 / 16;
    for (int idx = threadIdx.x; idx < BM * CH; idx += 64 * NW) {
      const int r = idx / CH, ch = idx - r * CH;
      store_out(reinterpret_cast<u32x4_t*>(C + static_cast<int64_t>(bm * BM + r) * ga.ldc + bn * BN * 2 + ch * 16),
                *reinterpret_cast<const u32x4_t*>(smem + cpos(r, ch * 16)));
    }
    __syncthreads();  // the next tile's loads overwrite the staging area
  }
  if (stage_t) {
    __syncthreads();
    // transposed tile rows (BM bf16 = BM*2 bytes each) -> CT, 16 bytes a thread
    constexpr int CH = BM * 2 / 16;
    for (int idx = threadIdx.x; idx < BN * CH; idx += 64 * NW) {
      const int c = idx / CH, ch = idx - c * CH;
      const char* src = smem + c * TST + ch * 16;
      const uint2 lo = *reinterpret_cast<const uint2*>(src);
      const uint2 hi = *reinterpret_cast<const uint2*>(src + 8);
      store_out(reinterpret_cast<u32x4_t*>(CT + static_cast<int64_t>(bn * BN + c) * ga.ldct + bm * BM * 2 + ch * 16),
                u32x4_t{lo.x, lo.y, hi.x, hi.y});
    }
    __syncthreads();  // the next tile's loads overwrite the staging area
  }
}


// Persistent launch: one workgroup per CU slot loops over tiles in rounds.
// Workgroup b runs on XCD b % 8; in round r the XCD's workgroups take the
// contiguous logical range r*G + (b % 8)*(G/8) + [0, G/8), i.e. a compact
// block of the banded order, and start it together, so the tiles of a block
// stay in step and share each operand slab through the XCD's L2.
template <int EPI, class Cfg>
__global__ __launch_bounds__(64 * Cfg::NW) __attribute__((amdgpu_waves_per_eu(Cfg::WPE, Cfg::WPE)))
void k_gemm_tile(GemmArgs ga) {
  // epilogue staging: the output tile (direct rows) or the mirrored tile
  constexpr int STAGED_C = Cfg::BM * Cfg::BN * 2, STAGED_T = Cfg::BN * (Cfg::BM * 2 + 8);
  constexpr int STAGED = STAGED_C > STAGED_T ? STAGED_C : STAGED_T;
  static_assert(STAGED <= 160 * 1024, "LDS budget");
  __shared__ __attribute__((aligned(1024))) char smem[Cfg::LDS > STAGED ? Cfg::LDS : STAGED];
  const int G = static_cast<int>(gridDim.x), b = static_cast<int>(blockIdx.x);
  for (int r = 0;; ++r) {
    const int logical = (G % 8 == 0) ? r * G + (b & 7) * (G / 8) + (b >> 3) : r * G + b;
    if (logical >= ga.total_tiles) break;
    int mat, bm, bn;
    tile_from_logical(ga, logical, mat, bm, bn);
    gemm_tile_body<EPI, Cfg>(ga, smem, mat, bm, bn);
  }
}

// One launch over the tiles of several chunks (a group): the product of
// the same Newton-Schulz step for every chunk, each with its own arguments.
// Tiles are numbered chunk by chunk (start[c] is chunk c's first), and the
// rounds run as in k_gemm_tile, so a tile of one chunk and a tile of the
// next can share a round.  Each tile's arithmetic is that of k_gemm_tile.
constexpr int kMaxGroup = 8;
struct GroupArgs {
  GemmArgs ga[kMaxGroup];
  int32_t start[kMaxGroup + 1];
  int32_t n;
};
static_assert(sizeof(GroupArgs) <= 4096, "kernel argument size");

template <int EPI, class Cfg>
__global__ __launch_bounds__(64 * Cfg::NW) __attribute__((amdgpu_waves_per_eu(Cfg::WPE, Cfg::WPE)))
void k_gemm_group(GroupArgs gr) {
  constexpr int STAGED_C = Cfg::BM * Cfg::BN * 2, STAGED_T = Cfg::BN * (Cfg::BM * 2 + 8);
  constexpr int STAGED = STAGED_C > STAGED_T ? STAGED_C : STAGED_T;
  __shared__ __attribute__((aligned(1024))) char smem[Cfg::LDS > STAGED ? Cfg::LDS : STAGED];
  const int G = static_cast<int>(gridDim.x), b = static_cast<int>(blockIdx.x);
  const int total = gr.start[gr.n];
  for (int r = 0;; ++r) {
    const int logical = (G % 8 == 0) ? r * G + (b & 7) * (G / 8) + (b >> 3) : r * G + b;
    if (logical >= total) break;
    int c = 0;
    while (c + 1 < gr.n && logical >= gr.start[c + 1]) ++c;
    const GemmArgs& ga = gr.ga[c];
    int mat, bm, bn;
    tile_from_logical(ga, logical - gr.start[c], mat, bm, bn);
    gemm_tile_body<EPI, Cfg>(ga, smem, mat, bm, bn);
  }
}

// Update from X0 when K = 0: O is X0 in the caller's layout (the direct
// buffer), one thread per element of the u-domain; grid = (ceil(rows*cols /
// 256), matrices).
template <typename XT>
__global__ __launch_bounds__(256) void k_apply_x0(const MatDesc* __restrict__ desc, ChunkGeom cg,
                                                  const XT* __restrict__ X, const XT* __restrict__ XTb,
                                                  const float* __restrict__ xscale, int final_kind) {
  const int m = blockIdx.y;
  const MatDesc md = desc[m];
  const int64_t numel = static_cast<int64_t>(md.rows) * md.cols;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= numel) return;
  const int64_t ur = i / md.cols, uc = i - ur * md.cols;
  const int64_t matX = static_cast<int64_t>(cg.S) * cg.L;
  const XT* D = (md.transposed ? XTb : X) + m * matX;
  const int ldD = md.transposed ? cg.S : cg.L;
  const float o = to_f32<XT>(D[ur * ldD + uc]) * xscale[m];  // X0 = r X~ (or X0 itself, scale 1)
  const int64_t w = view_index(md, ur, uc);
  if (final_kind == 0) {
    const float wv = load_as_f32(md.W, w, cg.param_dtype);
    store_from_f32(md.W, w, cg.param_dtype, fmaf(md.decay, wv, -md.upd_scale * o));
  } else {
    store_from_f32(md.out, w, cg.param_dtype, o);
  }
}

// ---------------------------------------------------------------------------
// Host-side launch sequence for one chunk.
// ---------------------------------------------------------------------------
#ifndef MUON_PERSISTENT
#define MUON_PERSISTENT 1
#endif

// Compute units of the current device (queried once per device).
int device_cu_count() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

template <class Cfg>
hipError_t launch_tile(int epi, GemmArgs ga, int nmat, hipStream_t st) {
  // ga arrives in 128 x 128 tiles and 128-byte slabs
  ga.tiles_m = ga.tiles_m * kTile / Cfg::BM;
  ga.tiles_n = ga.tiles_n * kTile / Cfg::BN;
  ga.tiles_per_mat = ga.syrk ? ga.tiles_m * (ga.tiles_m + 1) / 2 : ga.tiles_m * ga.tiles_n;
  ga.k_slabs = ga.k_slabs * 128 / Cfg::SLAB;
  ga.total_tiles = ga.tiles_per_mat * nmat;
  // B = b A + c A^2 = c (A^2 + (b/c) A): the A term joins the accumulators
  // in the main loop unless c = 0
  if (epi == EPI_POLY && ga.beta != 0.f) {
    ga.e_loop = 1;
    ga.alpha = ga.alpha / ga.beta;
  }
  // one workgroup per CU slot (persistent), never more workgroups than tiles
  const int slots = device_cu_count() * (160 * 1024 / Cfg::LDS);
  const int g = MUON_PERSISTENT ? min(ga.total_tiles, slots) : ga.total_tiles;
  const dim3 grid(static_cast<unsigned>(g)), block(64 * Cfg::NW);
  switch (epi) {
    case EPI_GRAM: hipLaunchKernelGGL((k_gemm_tile<EPI_GRAM, Cfg>), grid, block, 0, st, ga); break;
    case EPI_POLY: hipLaunchKernelGGL((k_gemm_tile<EPI_POLY, Cfg>), grid, block, 0, st, ga); break;
    case EPI_UPDATE: hipLaunchKernelGGL((k_gemm_tile<EPI_UPDATE, Cfg>), grid, block, 0, st, ga); break;
    default: {
      const bool o = ga.final_kind != 0, f32 = ga.param_dtype == DT_F32;
      if (!o && !f32) hipLaunchKernelGGL((k_gemm_tile<EPI_FINAL_W_BF16, Cfg>), grid, block, 0, st, ga);
      else if (!o) hipLaunchKernelGGL((k_gemm_tile<EPI_FINAL_W_F32, Cfg>), grid, block, 0, st, ga);
      else if (!f32) hipLaunchKernelGGL((k_gemm_tile<EPI_FINAL_O_BF16, Cfg>), grid, block, 0, st, ga);
      else hipLaunchKernelGGL((k_gemm_tile<EPI_FINAL_O_F32, Cfg>), grid, block, 0, st, ga);
      break;
    }
  }
  return hipGetLastError();
}

// The products of one step for a group of chunks on the 256 x 256 kernel:
// each chunk's arguments prepared as launch_tile prepares them, one
// persistent launch over all their tiles.  The chunks share the product, the
// final kind and the parameter dtype.
template <class Cfg>
hipError_t launch_group(int epi, const GemmArgs* gas, const int* nmats, int n, hipStream_t st) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  GroupArgs gr{};
  gr.n = n;
  gr.start[0] = 0;
  for (int c = 0; c < n; ++c) {
    GemmArgs ga = gas[c];
    ga.tiles_m = ga.tiles_m * kTile / Cfg::BM;
    ga.tiles_n = ga.tiles_n * kTile / Cfg::BN;
    ga.tiles_per_mat = ga.syrk ? ga.tiles_m * (ga.tiles_m + 1) / 2 : ga.tiles_m * ga.tiles_n;
    ga.k_slabs = ga.k_slabs * 128 / Cfg::SLAB;
    ga.total_tiles = ga.tiles_per_mat * nmats[c];
    if (epi == EPI_POLY && ga.beta != 0.f) {
      ga.e_loop = 1;
      ga.alpha = ga.alpha / ga.beta;
    }
    if (c > 0 && (ga.final_kind != gr.ga[0].final_kind || ga.param_dtype != gr.ga[0].param_dtype))
      return hipErrorInvalidValue;
    gr.ga[c] = ga;
    gr.start[c + 1] = gr.start[c] + ga.total_tiles;
  }
  const int total = gr.start[n];
  const int slots = device_cu_count() * (160 * 1024 / Cfg::LDS);
  const dim3 grid(static_cast<unsigned>(min(total, slots))), block(64 * Cfg::NW);
  switch (epi) {
    case EPI_GRAM: hipLaunchKernelGGL((k_gemm_group<EPI_GRAM, Cfg>), grid, block, 0, st, gr); break;
    case EPI_POLY: hipLaunchKernelGGL((k_gemm_group<EPI_POLY, Cfg>), grid, block, 0, st, gr); break;
    case EPI_UPDATE: hipLaunchKernelGGL((k_gemm_group<EPI_UPDATE, Cfg>), grid, block, 0, st, gr); break;
    default: {
      const bool o = gr.ga[0].final_kind != 0, f32 = gr.ga[0].param_dtype == DT_F32;
      if (!o && !f32) hipLaunchKernelGGL((k_gemm_group<EPI_FINAL_W_BF16, Cfg>), grid, block, 0, st, gr);
      else if (!o) hipLaunchKernelGGL((k_gemm_group<EPI_FINAL_W_F32, Cfg>), grid, block, 0, st, gr);
      else if (!f32) hipLaunchKernelGGL((k_gemm_group<EPI_FINAL_O_BF16, Cfg>), grid, block, 0, st, gr);
      else hipLaunchKernelGGL((k_gemm_group<EPI_FINAL_O_F32, Cfg>), grid, block, 0, st, gr);
      break;
    }
  }
  return hipGetLastError();
}

// The 256 x 256 kernel runs the bf16 products whose padded extents are
// multiples of 256 (and whose rows fit its offsets): the symmetric ones when
// S is, the update ones (which read X through transposing LDS reads) when S
// and L are.  Everything else runs on the 128 x 128 kernel, whose update
// reads X^T and whose offsets are 64-bit.
template <typename T>
hipError_t launch_gemm(int epi, GemmArgs ga, int nmat, hipStream_t st) {
  if (sizeof(T) == 2 && ga.tiles_m % 2 == 0 && ga.syrk && ga.ldp < kTileMaxRowBytes &&
      ga.ldq < kTileMaxRowBytes && (!ga.E || ga.lde < kTileMaxRowBytes))
    return launch_tile<CfgSquare>(epi, ga, nmat, st);
  const dim3 grid(static_cast<unsigned>(ga.tiles_per_mat) * nmat), block(256);
  switch (epi) {
    case EPI_GRAM: hipLaunchKernelGGL((k_gemm_nt<T, EPI_GRAM>), grid, block, 0, st, ga); break;
    case EPI_POLY: hipLaunchKernelGGL((k_gemm_nt<T, EPI_POLY>), grid, block, 0, st, ga); break;
    case EPI_UPDATE: hipLaunchKernelGGL((k_gemm_nt<T, EPI_UPDATE>), grid, block, 0, st, ga); break;
    default: hipLaunchKernelGGL((k_gemm_nt<T, EPI_FINAL>), grid, block, 0, st, ga); break;
  }
  return hipGetLastError();
}

// Brackets one launch with the optional timer.
struct Timed {
  LaunchTimer* t;
  int kind;
  hipStream_t st;
  Timed(LaunchTimer* timer, int k, hipStream_t s) : t(timer), kind(k), st(s) {
    if (t) t->begin(kind, st);
  }
  void done(double flops, double exec_flops, double bytes) {
    if (t) t->end(kind, st, flops, exec_flops, bytes);
  }
};

// ---------------------------------------------------------------------------
// Fused Newton-Schulz for short sides up to 128 (k_ns_small): the whole step
// of a chunk -- momentum, norm, X0, every Newton-Schulz step and the update --
// in one launch.  Such matrices are far too small for the tile kernels: a
// 128 x 256 fp32 product fills one or two workgroups, so separate launches
// leave the device idle and each product runs on a single compute unit.
//
// Each matrix is taken by a group of G = RB x CB workgroups: RB row blocks
// of 32 rows of X (the padded short side Sx = 32 RB) times CB column groups
// (a function of the shape alone, so results do not depend on the batch).
// Per step, every product on MFMA in 16 x 16 units shared out over the four
// wavefronts:
//   A[Ri, Cc] = X[Ri, :] X[Cc, :]^T             column blocks c = j, j + CB, ..
//   -- group barrier --
//   B[Ri, Cc] = b A[Ri, Cc] + c A[Ri, :] A[Cc, :]^T   (A symmetric)
//   -- group barrier (CB > 1: rows Ri of B come from several workgroups) --
//   X'[Ri, Dd] = a X[Ri, Dd] + B[Ri, :] X^T[Dd, :]^T  column blocks d = j, j + CB, ..
//   -- group barrier --
// X is kept in both orientations, so every operand is a row-major matrix
// with K contiguous, stored tiled (see ti).  The prologue writes u itself
// into X and applies r = 1 / (||u|| + eps) in the first step's products
// (exact fp32 u; X0 = r u is formed first when r is far from 1).  The last
// step writes W (or the output) straight from the fp32 values, in the
// parameter's own layout.  Extents are padded to multiples of 32; the
// padding of X, A and B is written as zeros and stays zero.
//
// The members of a group run on one XCD (workgroup b runs on XCD b % 8, and
// each workgroup checks its XCC_ID against its group's): their data meets in
// that XCD's L2, so a barrier drains the memory operations of every wave and
// bumps a counter, and every read of data that other members wrote is a
// non-temporal load, which bypasses the compute unit's own (incoherent) L1.
// Should a group find its members spread over XCDs, every barrier of that
// group also writes back and invalidates at device scope.  Spins are
// bounded, so every wave ends whatever happens.
// ---------------------------------------------------------------------------
struct SmallArgs {
  const MatDesc* desc;
  StepScalars sc;
  int32_t s, l, S, L, Sx, Lx;
  int32_t nmat, G, RB, CB, groups, K;
  int32_t param_dtype;
  char* X[2];
  char* XT[2];
  char* A;
  char* B;
  int64_t matX, matA;        // bytes per matrix
  double* partials;          // nmat x kSmallMaxGroup
  unsigned* sync;            // per group: [0] counter, [1] spin timeouts, [2 .. 2 + G) member XCC ids
  float coeffs[3 * 64];      // (a, b, c) per step
};

__device__ __forceinline__ unsigned xcc_id() {
  return __builtin_amdgcn_s_getreg((3 << 11) | (0 << 6) | 20) & 15u;  // HW_REG_XCC_ID, bits [3:0]
}

__device__ __forceinline__ void group_barrier(unsigned* sync, unsigned target, bool local) {
  __builtin_amdgcn_s_waitcnt(0);  // this wave's loads and stores are done (stores reached L2)
  __syncthreads();
  if (threadIdx.x == 0) {
    if (!local) __threadfence();
    __hip_atomic_fetch_add(sync, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    unsigned spins = 0;
    while (__hip_atomic_load(sync, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      __builtin_amdgcn_s_sleep(2);
      if (++spins > (1u << 22)) {  // never expected: count it and go on
        __hip_atomic_fetch_add(sync + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
    }
    if (!local) __atomic_thread_fence(__ATOMIC_ACQUIRE);
  }
  __syncthreads();
}

// Loads of data other members wrote: non-temporal, so they never allocate, and
// never hit, a line in this compute unit's L1, which is not coherent with
// the other compute units (measured: plain loads after the barrier return
// stale L1 lines; non-temporal ones do not).  The L2 they read is the one
// the writers' stores reached.
__device__ __forceinline__ u32x4_t ld16(const char* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
}

typedef float f32x4_t __attribute__((ext_vector_type(4)));

// 16 x 16 blocks of P Q^T (fp32), K in k-groups of 16 elements (64 bytes of a
// row).  Lane l loads the 16 bytes of row l % 16 at byte 16 (l / 16) of a
// group and issues four v_mfma_f32_16x16x4_f32, the j-th taking element j
// (k = j, 4 + j, 8 + j, 12 + j across the lanes' four row quarters); even
// and odd groups accumulate apart and are added at the end of the block.
// Result layout: lane l, register r holds row 4 (l / 16) + r, column l % 16.
//
// small_units runs the 16 x 16 units of one phase, shared out round-robin
// over the four wavefronts.  unit(u, P, Q, row0, col0) gives unit u's
// operands (the first chunks of its 16-row blocks, tiled layout) and origin; pre(row, col) is loaded
// with the unit's first operands; epi(row, col, value, term) receives the 4
// values of each lane.  A wavefront's units and their K batches form one
// stream: the loads of the next batch (of the same or the next unit) are in
// flight while the MFMAs of the current one issue.
constexpr int kSmallBatch = 8;  // k-groups per batch
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// The fused launch keeps X, X^T, A and B in a tiled layout: each 16-row x
// 16-k chunk of a row-major matrix is 1 KB, stored in the order of the lanes
// that take it as an MFMA operand (lane l: row l % 16, k 4 (l / 16) .. + 3),
// chunks row-block major.  A wavefront's operand load is then 1 KB of
// consecutive bytes (whole cache lines), where the row-major layout touched
// 16 lines for 64 bytes each (measured 4x slower).  Element (r, k) of a
// matrix with kg k-groups per row, in floats:
__device__ __forceinline__ int64_t ti(int r, int k, int kg) {
  return (static_cast<int64_t>(r >> 4) * kg + (k >> 4)) * 256 + (((k & 15) >> 2) * 16 + (r & 15)) * 4 + (k & 3);
}
// The bf16 form: 16-row x 32-k chunks of 1 KB (lane l: row l % 16,
// k 8 (l / 16) .. + 7, the operand of v_mfma_f32_16x16x32_bf16), kg k-groups
// of 32 per row, in elements.
__device__ __forceinline__ int64_t ti_b(int r, int k, int kg) {
  return (static_cast<int64_t>(r >> 4) * kg + (k >> 5)) * 512 + (((k & 31) >> 3) * 16 + (r & 15)) * 8 + (k & 7);
}
template <typename XT>
__device__ __forceinline__ int64_t tix(int r, int k, int kg) {
  if constexpr (sizeof(XT) == 2) return ti_b(r, k, kg);
  else return ti(r, k, kg);
}

template <typename XT, typename Unit, typename Pre, typename Epi>
__device__ __forceinline__ void small_units(int nunits, int kg, Unit&& unit, Pre&& pre, Epi&& epi) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int mine = nunits > wave ? (nunits - wave + 3) / 4 : 0;  // this wavefront's units
  const int nbat = (kg + kSmallBatch - 1) / kSmallBatch;
  const int total = mine * nbat;
  if (total == 0) return;
  struct Batch {
    u32x4_t a[kSmallBatch], b[kSmallBatch];
    float term[4];
  };
  // the operands of stream item `it` (unit it / nbat, batch it % nbat)
  auto issue = [&](int it, Batch& bt) __attribute__((always_inline)) {
    const int u = wave + 4 * (it / nbat), bb = it % nbat;
    const char* P;
    const char* Q;
    int row0, col0;
    unit(u, P, Q, row0, col0);
    const char* pr = P + lane * 16;
    const char* qr = Q + lane * 16;
    const int g0 = bb * kSmallBatch;
#pragma unroll
    for (int t = 0; t < kSmallBatch; ++t)
      if (g0 + t < kg) {
        bt.a[t] = ld16(pr + static_cast<int64_t>(g0 + t) * 1024);
        bt.b[t] = ld16(qr + static_cast<int64_t>(g0 + t) * 1024);
      }
    if (bb == 0) {
      const int row = row0 + 4 * (lane >> 4), col = col0 + (lane & 15);
#pragma unroll
      for (int r = 0; r < 4; ++r) bt.term[r] = pre(row + r, col);
    }
  };
  f32x4_t acc[2];
  float term[4];
  auto consume = [&](int it, Batch& bt) __attribute__((always_inline)) {
    const int bb = it % nbat, g0 = bb * kSmallBatch;
    if (bb == 0) {
      acc[0] = acc[1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int r = 0; r < 4; ++r) term[r] = bt.term[r];
    }
#pragma unroll
    for (int t = 0; t < kSmallBatch; ++t)
      if (g0 + t < kg) {
        if constexpr (sizeof(XT) == 2) {
          acc[t & 1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, bt.a[t]),
                                                               __builtin_bit_cast(bf16x8_t, bt.b[t]), acc[t & 1], 0, 0, 0);
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[t & 1] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bt.a[t][j]), __uint_as_float(bt.b[t][j]),
                                                              acc[t & 1], 0, 0, 0);
        }
      }
    if (bb == nbat - 1) {
      const int u = wave + 4 * (it / nbat);
      const char* P;
      const char* Q;
      int row0, col0;
      unit(u, P, Q, row0, col0);
      const f32x4_t v = acc[0] + acc[1];
      const int row = row0 + 4 * (lane >> 4), col = col0 + (lane & 15);
#pragma unroll
      for (int r = 0; r < 4; ++r) epi(row + r, col, v[r], term[r]);
    }
  };
  Batch b0, b1;
  issue(0, b0);
  for (int it = 0; it < total; it += 2) {
    if (it + 1 < total) issue(it + 1, b1);
    consume(it, b0);
    if (it + 1 >= total) break;
    if (it + 2 < total) issue(it + 2, b0);
    consume(it + 1, b1);
  }
}

template <typename T>
__device__ __forceinline__ void put(char* base, int64_t idx, float v) {
  reinterpret_cast<T*>(base)[idx] = from_f32<T>(v);
}
template <typename T>
__device__ __forceinline__ float get(const char* base, int64_t idx) {
  return to_f32<T>(__builtin_nontemporal_load(reinterpret_cast<const T*>(base) + idx));
}

// XT: float (fp32 Newton-Schulz, X exact u) or uint16_t (bf16: X, A and B
// stored as bfloat16 between the products, fp32 accumulation).
template <typename GT, typename XT, bool MOM>
__global__ __launch_bounds__(256) void k_ns_small(SmallArgs sa) {
  constexpr int KG = sizeof(XT) == 2 ? 32 : 16;  // k per operand chunk
  __shared__ double red4[4];
  const int b = blockIdx.x, xcd = b & 7, slot = b >> 3;
  const int group = (slot / sa.G) * 8 + xcd, member = slot % sa.G;
  const int bi = member / sa.CB, bj = member % sa.CB;  // row block, column group
  unsigned* const sync = sa.sync + group * 64;
  if (threadIdx.x == 0) __hip_atomic_store(sync + 2 + member, xcc_id(), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  unsigned nbar = 0;
  bool local = false;
  const int kgx = sa.L / KG, kgs = sa.S / KG;      // k-groups per row of X, of X^T, A and B
  const int ncb = sa.Lx / 32;                                    // column blocks of X
  const int c0 = bj * ncb / sa.CB, c1 = (bj + 1) * ncb / sa.CB;  // this member's, in the prologue
  const int w = (c1 - c0) * 32;                                  // prologue columns of this member
  const float beta = sa.sc.beta, omb = sa.sc.one_minus_beta;
  for (int m = group; m < sa.nmat; m += sa.groups) {
    const MatDesc md = sa.desc[m];
    const bool tr = md.transposed != 0;
    const GT* g = static_cast<const GT*>(md.g);
    char* X0 = sa.X[0] + m * sa.matX;
    char* XT0 = sa.XT[0] + m * sa.matX;
    // element e of the member's 32 x w block of X: consecutive threads on
    // consecutive elements of u's rows (coalesced for either orientation)
    auto coord = [&](int e, int& xr, int& xc) {
      if (tr) { xr = bi * 32 + (e & 31); xc = c0 * 32 + (e >> 5); }
      else { xr = bi * 32 + e / w; xc = c0 * 32 + e % w; }
    };
    // ---- prologue pass 1: momentum, u into X (fp32, exact), sum of u^2 ----
    double acc2 = 0.0;
    const int ne = 32 * w;
    for (int e0 = threadIdx.x; e0 < ne; e0 += 256 * 8) {
      float gv[8], bv[8];
      int64_t gi[8], bix[8];
      bool in[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        int xr, xc;
        coord(e0 + 256 * t, xr, xc);
        in[t] = e0 + 256 * t < ne && xr < sa.s && xc < sa.l;
        const int ur = tr ? xc : xr, uc = tr ? xr : xc;
        gi[t] = in[t] ? view_index(md, ur, uc) : 0;
        bix[t] = (MOM && in[t]) ? buf_index(md, ur, uc) : 0;
        gv[t] = in[t] ? to_f32<GT>(g[gi[t]]) : 0.f;
        bv[t] = (MOM && in[t]) ? md.buf[bix[t]] : 0.f;
      }
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        if (e0 + 256 * t >= ne) continue;
        float u = gv[t];
        if (MOM && in[t]) {
          const float bn = fmaf(beta, bv[t], omb * gv[t]);
          md.buf[bix[t]] = bn;
          u = sa.sc.nesterov ? fmaf(beta, bn, omb * gv[t]) : bn;
        }
        acc2 = fma(static_cast<double>(u), static_cast<double>(u), acc2);
        int xr, xc;
        coord(e0 + 256 * t, xr, xc);
        put<XT>(X0, tix<XT>(xr, xc, kgx), u);
        put<XT>(XT0, tix<XT>(xc, xr, kgs), u);
      }
    }
    const double part = block_sum_256(acc2, red4);
    if (threadIdx.x == 0) sa.partials[static_cast<int64_t>(m) * kSmallMaxGroup + member] = part;
    ++nbar;
    group_barrier(sync, nbar * sa.G, local);
    if (nbar == 1) {  // the members' XCDs are known from here on
      bool same = true;
      for (int q = 0; q < sa.G; ++q)
        same = same && __hip_atomic_load(sync + 2 + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                           __hip_atomic_load(sync + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      local = same;
    }
    double nsq = 0.0;
    for (int q = 0; q < sa.G; ++q)
      nsq += __builtin_nontemporal_load(sa.partials + static_cast<int64_t>(m) * kSmallMaxGroup + q);
    const double r = 1.0 / (sqrt(nsq) + static_cast<double>(sa.sc.eps));
    // X holds u itself (exact in fp32).  While r keeps (r u)(r u)^T far
    // inside the fp32 range, the first step applies it (A0 = r^2 u u^T,
    // X1 = r (a u + B0 u)); otherwise, and for K = 0, X0 = r u is formed here.
    const bool fold = sa.K > 0 && r >= 0x1p-40 && r <= 0x1p40;
    const float xs = fold ? static_cast<float>(r) : 1.f;
    float s1, s2;
    split_scale(r, s1, s2);
    // ---- prologue pass 2 (unless folded): X0 = r u over the member's block ----
    if (!fold)
    for (int e0 = threadIdx.x; e0 < ne; e0 += 256 * 8) {
      float v[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        int xr, xc;
        coord(e0 + 256 * t, xr, xc);
        float u = 0.f;
        if (e0 + 256 * t < ne) {
          if constexpr (sizeof(XT) == 4) {
            u = get<XT>(X0, tix<XT>(xr, xc, kgx));  // u itself, exact
          } else if (xr < sa.s && xc < sa.l) {
            // X holds u rounded to bf16: form u again from g and the advanced
            // momentum (this thread's own writes), so r u is rounded once
            const int ur = tr ? xc : xr, uc = tr ? xr : xc;
            const float gv = to_f32<GT>(g[view_index(md, ur, uc)]);
            u = gv;
            if (MOM) {
              const float bn = md.buf[buf_index(md, ur, uc)];
              u = sa.sc.nesterov ? fmaf(beta, bn, omb * gv) : bn;
            }
          }
        }
        v[t] = (u * s1) * s2;
      }
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        if (e0 + 256 * t >= ne) continue;
        int xr, xc;
        coord(e0 + 256 * t, xr, xc);
        if (sa.K == 0) {
          if (xr < sa.s && xc < sa.l) {
            const int64_t pidx = view_index(md, tr ? xc : xr, tr ? xr : xc);
            if (sa.sc.final_kind == 0)
              store_from_f32(md.W, pidx, sa.param_dtype,
                             fmaf(md.decay, load_as_f32(md.W, pidx, sa.param_dtype), -md.upd_scale * v[t]));
            else
              store_from_f32(md.out, pidx, sa.param_dtype, v[t]);
          }
        } else {
          put<XT>(X0, tix<XT>(xr, xc, kgx), v[t]);
          put<XT>(XT0, tix<XT>(xc, xr, kgs), v[t]);
        }
      }
    }
    if (sa.K == 0) continue;
    if (!fold) {
      ++nbar;
      group_barrier(sync, nbar * sa.G, local);
    }
    int cur = 0;
    const int na = (sa.RB - bj + sa.CB - 1) / sa.CB;      // 32-column blocks of A and B of this member
    for (int k = 0; k < sa.K; ++k) {
      const float ca = sa.coeffs[3 * k], cb = sa.coeffs[3 * k + 1], cc = sa.coeffs[3 * k + 2];
      const float sa_ = k == 0 ? xs * xs : 1.f, sx_ = k == 0 ? xs : 1.f;  // the folded r on the first step
      const char* Xc = sa.X[cur] + m * sa.matX;
      const char* XTc = sa.XT[cur] + m * sa.matX;
      char* Am = sa.A + m * sa.matA;
      char* Bm = sa.B + m * sa.matA;
      // unit u of a phase over 32 x 32 blocks: block u / 4, quarter u % 4
      // A = X X^T: rows bi, column blocks bj, bj + CB, ..
      small_units<XT>(
          4 * na, sa.Lx / KG,
          [&](int u, const char*& P, const char*& Q, int& row0, int& col0) {
            row0 = bi * 32 + 16 * ((u & 3) >> 1);
            col0 = (bj + (u >> 2) * sa.CB) * 32 + 16 * (u & 1);
            P = Xc + tix<XT>(row0, 0, kgx) * static_cast<int64_t>(sizeof(XT));
            Q = Xc + tix<XT>(col0, 0, kgx) * static_cast<int64_t>(sizeof(XT));
          },
          [](int, int) { return 0.f; },
          [&](int row, int col, float v, float) { put<XT>(Am, tix<XT>(row, col, kgs), sa_ * v); });
      ++nbar;
      group_barrier(sync, nbar * sa.G, local);
      // B = b A + c A A (A symmetric: column block c of A is row block c)
      small_units<XT>(
          4 * na, sa.Sx / KG,
          [&](int u, const char*& P, const char*& Q, int& row0, int& col0) {
            row0 = bi * 32 + 16 * ((u & 3) >> 1);
            col0 = (bj + (u >> 2) * sa.CB) * 32 + 16 * (u & 1);
            P = Am + tix<XT>(row0, 0, kgs) * static_cast<int64_t>(sizeof(XT));
            Q = Am + tix<XT>(col0, 0, kgs) * static_cast<int64_t>(sizeof(XT));
          },
          [&](int row, int col) { return get<XT>(Am, tix<XT>(row, col, kgs)); },
          [&](int row, int col, float v, float a_) { put<XT>(Bm, tix<XT>(row, col, kgs), fmaf(cb, a_, cc * v)); });
      if (sa.CB > 1) {
        ++nbar;
        group_barrier(sync, nbar * sa.G, local);
      }
      // X' = a X + B X: rows bi, column blocks bj, bj + CB, .. of X
      const bool last = k + 1 == sa.K;
      char* Xn = sa.X[cur ^ 1] + m * sa.matX;
      char* XTn = sa.XT[cur ^ 1] + m * sa.matX;
      const int nx = (ncb - bj + sa.CB - 1) / sa.CB;
      small_units<XT>(
          4 * nx, sa.Sx / KG,
          [&](int u, const char*& P, const char*& Q, int& row0, int& col0) {
            row0 = bi * 32 + 16 * ((u & 3) >> 1);
            col0 = (bj + (u >> 2) * sa.CB) * 32 + 16 * (u & 1);
            P = Bm + tix<XT>(row0, 0, kgs) * static_cast<int64_t>(sizeof(XT));
            Q = XTc + tix<XT>(col0, 0, kgs) * static_cast<int64_t>(sizeof(XT));
          },
          [&](int row, int col) { return get<XT>(Xc, tix<XT>(row, col, kgx)); },
          [&](int xr, int xc, float v, float x_) {
            const float o = sx_ * fmaf(ca, x_, v);
            if (!last) {
              put<XT>(Xn, tix<XT>(xr, xc, kgx), o);
              put<XT>(XTn, tix<XT>(xc, xr, kgs), o);
            } else if (xr < sa.s && xc < sa.l) {
              const int64_t pidx = view_index(md, tr ? xc : xr, tr ? xr : xc);
              if (sa.sc.final_kind == 0)
                store_from_f32(md.W, pidx, sa.param_dtype,
                               fmaf(md.decay, load_as_f32(md.W, pidx, sa.param_dtype), -md.upd_scale * o));
              else
                store_from_f32(md.out, pidx, sa.param_dtype, o);
            }
          });
      if (!last) {
        ++nbar;
        group_barrier(sync, nbar * sa.G, local);
      }
      cur ^= 1;
    }
  }
}

// Zeroes n words (the group counters before a fused launch).
__global__ __launch_bounds__(256) void k_zero_words(unsigned* p, int n) {
  for (int i = threadIdx.x; i < n; i += 256) p[i] = 0u;
}

template <typename GT, typename XT>
hipError_t run_small(const ChunkGeom& cg, const MatDesc* d_desc, const ChunkBuffers& wb, const StepScalars& sc,
                     const float* coeffs, int K, hipStream_t st, LaunchTimer* timer) {
  SmallArgs sa{};
  sa.desc = d_desc;
  sa.sc = sc;
  sa.s = cg.s; sa.l = cg.l; sa.S = cg.S; sa.L = cg.L;
  sa.Sx = (cg.s + 31) / 32 * 32;
  sa.Lx = (cg.l + 31) / 32 * 32;
  sa.nmat = cg.nmat;
  sa.RB = sa.Sx / 32;
  const int cus = device_cu_count();
  // column groups: 4, or as many as there are 32-column blocks of X.  A
  // function of the shape alone, so that the order of every sum, and with
  // it each matrix's result, does not depend on the other matrices of the call.
  sa.CB = min(4, sa.Lx / 32);
  sa.G = sa.RB * sa.CB;
  // groups: 8 per round (one per XCD), as many rounds as fit one workgroup per CU
  const int rounds = max(1, min((cg.nmat + 7) / 8, cus / (8 * sa.G)));
  sa.groups = 8 * rounds;
  sa.K = K;
  sa.param_dtype = cg.param_dtype;
  sa.X[0] = static_cast<char*>(wb.X[0]); sa.X[1] = static_cast<char*>(wb.X[1]);
  sa.XT[0] = static_cast<char*>(wb.XT[0]); sa.XT[1] = static_cast<char*>(wb.XT[1]);
  sa.A = static_cast<char*>(wb.A); sa.B = static_cast<char*>(wb.B);
  sa.matX = static_cast<int64_t>(cg.S) * cg.L * sizeof(XT);
  sa.matA = static_cast<int64_t>(cg.S) * cg.S * sizeof(XT);
  sa.partials = wb.partials;
  sa.sync = wb.sync;
  for (int i = 0; i < 3 * K; ++i) sa.coeffs[i] = coeffs[i];
  Timed tm(timer, KK_SMALL, st);
  hipLaunchKernelGGL(k_zero_words, dim3(1), dim3(256), 0, st, wb.sync, sa.groups * 64);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 grid(static_cast<unsigned>(sa.groups * sa.G));
  if (sc.momentum)
    hipLaunchKernelGGL((k_ns_small<GT, XT, true>), grid, dim3(256), 0, st, sa);
  else
    hipLaunchKernelGGL((k_ns_small<GT, XT, false>), grid, dim3(256), 0, st, sa);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const double nm = cg.nmat, s = cg.s, l = cg.l, Sx = sa.Sx, Lx = sa.Lx;
  const double gsz = sizeof(GT), psz = cg.param_dtype == DT_BF16 ? 2.0 : 4.0;
  tm.done(nm * K * (4.0 * s * s * l + 2.0 * s * s * s), nm * K * (4.0 * Sx * Sx * Lx + 2.0 * Sx * Sx * Sx),
          nm * s * l * (gsz + (sc.momentum ? 8.0 : 0.0) + (sc.final_kind == 0 ? 2.0 * psz : psz)));
  return hipSuccess;
}

template <typename GT, typename XT>
hipError_t run_prologue_t(const ChunkGeom& cg, const MatDesc* d_desc, const ChunkBuffers& wb,
                       const StepScalars& sc, const float* coeffs, int K, hipStream_t st,
                       LaunchTimer* timer) {
  const int nmat = cg.nmat;
  const double nm = nmat;
  const int64_t numel = static_cast<int64_t>(cg.s) * cg.l;
  const double ne = double(numel);
  const int nparts = static_cast<int>(norm_tiles(cg.S, cg.L));
  const double gsz = sizeof(GT), xsz = sizeof(XT);
  const double psz = cg.param_dtype == DT_BF16 ? 2.0 : 4.0;
  // bf16 with S and L multiples of 256: the update products run on the
  // 256 x 256 kernel and read X through transposing LDS reads, so no X^T is
  // kept (K = 0 applies X0 from whichever layout matches the parameter).
  const bool qtr = !chunk_keeps_xt(cg.S, cg.L, sizeof(XT) == 4, K);
  XT* const xt0 = qtr ? nullptr : static_cast<XT*>(wb.XT[0]);
  hipError_t e;
  XT* const x0 = static_cast<XT*>(wb.X[0]);
  {
    Timed tm(timer, KK_PARTIALS, st);
    const dim3 grid(cg.L / 64, cg.S / 64, nmat);
    if (sc.momentum)
      hipLaunchKernelGGL((k_prologue<GT, XT, true>), grid, dim3(256), 0, st, d_desc, sc, cg, x0, xt0, wb.partials);
    else
      hipLaunchKernelGGL((k_prologue<GT, XT, false>), grid, dim3(256), 0, st, d_desc, sc, cg, x0, xt0, wb.partials);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // reads g (and the momentum), writes the momentum and X~ (and X~^T)
    tm.done(0, 0, nm * ne * (gsz + (sc.momentum ? 8.0 : 0.0) + (qtr ? 1.0 : 2.0) * xsz) + nm * nparts * 8.0);
  }
  {
    Timed tm(timer, KK_FINALIZE, st);
    hipLaunchKernelGGL(k_finalize, dim3(nmat), dim3(1024), 0, st, wb.partials, nparts, sc.eps, wb.rscale,
                       wb.xscale);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    tm.done(0, 0, nm * nparts * 8.0 + nm * 12.0);
  }
  {
    Timed tm(timer, KK_NORMALIZE, st);
    const dim3 grid(64, nmat);
    if (sc.momentum)
      hipLaunchKernelGGL((k_rescale<GT, XT, true>), grid, dim3(256), 0, st, d_desc, wb.rscale, wb.xscale, sc, cg,
                         x0, xt0);
    else
      hipLaunchKernelGGL((k_rescale<GT, XT, false>), grid, dim3(256), 0, st, d_desc, wb.rscale, wb.xscale, sc,
                         cg, x0, xt0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    tm.done(0, 0, nm * 12.0);  // nothing else unless a norm is out of range
  }

  if (K == 0) {
    Timed tm(timer, KK_APPLY_X0, st);
    const int64_t blocks = (numel + 255) / 256;
    hipLaunchKernelGGL((k_apply_x0<XT>), dim3(static_cast<unsigned>(blocks), nmat), dim3(256), 0, st,
                       d_desc, cg, static_cast<const XT*>(wb.X[0]), static_cast<const XT*>(wb.XT[0]),
                       wb.xscale, sc.final_kind);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    tm.done(0, 0, nm * ne * (xsz + (sc.final_kind == 0 ? 2.0 * psz : psz)));
    return hipSuccess;
  }
  return hipSuccess;
}

// The three products of Newton-Schulz step k of a chunk (after the
// prologue): their launch arguments and work accounting.  `cur` selects the
// iterate the step reads.
struct StepProducts {
  GemmArgs gram, poly, upd;
  bool last;              // upd is the last step's product (parameter update or O)
  double f[3], x[3], b[3];  // dense flops, executed flops, bytes of gram, poly, upd
};

template <typename XT>
StepProducts step_products(const ChunkGeom& cg, const MatDesc* d_desc, const ChunkBuffers& wb,
                           const StepScalars& sc, const float* coeffs, int K, int k, int cur) {
  const bool qtr = !chunk_keeps_xt(cg.S, cg.L, sizeof(XT) == 4, K);
  const double nm = cg.nmat;
  const double s = cg.s, l = cg.l;
  const double xsz = sizeof(XT);
  const double psz = cg.param_dtype == DT_BF16 ? 2.0 : 4.0;
  const int es = static_cast<int>(sizeof(XT));
  const int64_t matX = static_cast<int64_t>(cg.S) * cg.L * es;
  const int64_t matA = static_cast<int64_t>(cg.S) * cg.S * es;
  const int ts = cg.S / kTile, tl = cg.L / kTile;
  // Work accounting: `flops` is the dense count of each product on the real
  // extents (Eq. 1); `exec` is what the MFMAs execute: padded extents, and
  // for the symmetric products the upper tiles of the kernel that runs them
  // (256 x 256 tiles when bf16, S a multiple of 256 and the rows short
  // enough, else 128 x 128; see launch_gemm).
  auto upper_frac = [&](bool tile) {
    const int t = tile ? cg.S / 256 : ts;
    return double(t * (t + 1) / 2) / double(t * t);
  };
  const bool tile_sym = sizeof(XT) == 2 && cg.S % 256 == 0;
  const double gram_frac = upper_frac(tile_sym && tile_rows_fit(cg.S, cg.L, es));
  const double poly_frac = upper_frac(tile_sym && tile_rows_fit(cg.S, cg.S, es));
  const double Sp = cg.S, Lp = cg.L;
  StepProducts r{};
  const float a = coeffs[3 * k], b = coeffs[3 * k + 1], c = coeffs[3 * k + 2];
  const char* X = static_cast<const char*>(wb.X[cur]);
  const char* XTc = static_cast<const char*>(wb.XT[cur]);
  // A = X X^T: M = N = S, K = L.
  GemmArgs& g = r.gram;
  g.P = X; g.p_mat = matX; g.ldp = cg.L * es;
  g.Q = X; g.q_mat = matX; g.ldq = cg.L * es;
  g.k_slabs = cg.L * es / 128;
  g.tiles_m = ts; g.tiles_n = ts; g.syrk = 1; g.tiles_per_mat = ts * (ts + 1) / 2;
  g.C = static_cast<char*>(wb.A); g.c_mat = matA; g.ldc = cg.S * es;
  g.xscale = k == 0 ? wb.xscale : nullptr;  // A0 = r^2 X~ X~^T
  // Under qtr every consumer of A and B runs on the 256 x 256 kernel and
  // reads them as upper-triangle tiles (mode 1): no mirrored tile is
  // written.  Otherwise the lower triangle is written as the mirror.
  if (!qtr) { g.CT = g.C; g.ct_mat = matA; g.ldct = g.ldc; }
  r.f[0] = nm * 2 * s * s * l; r.x[0] = nm * 2 * Sp * Sp * Lp * gram_frac; r.b[0] = nm * (s * l + s * s) * xsz;
  // B = b A + c A A^T: M = N = K = S.
  GemmArgs& pp = r.poly;
  pp = g;
  pp.xscale = nullptr;
  pp.P = static_cast<const char*>(wb.A); pp.p_mat = matA; pp.ldp = cg.S * es;
  pp.Q = pp.P; pp.q_mat = matA; pp.ldq = pp.ldp;
  pp.k_slabs = cg.S * es / 128;
  pp.E = pp.P; pp.e_mat = matA; pp.lde = pp.ldp;
  pp.ET = pp.P; pp.et_mat = matA; pp.ldet = pp.ldp;  // A is symmetric
  pp.C = static_cast<char*>(wb.B); pp.CT = qtr ? nullptr : pp.C;
  pp.p_mode = pp.q_mode = qtr ? 1 : 0;
  pp.alpha = b; pp.beta = c;
  r.f[1] = nm * 2 * s * s * s; r.x[1] = nm * 2 * Sp * Sp * Sp * poly_frac; r.b[1] = nm * 2 * s * s * xsz;
  // X' = a X + B X: M = S, N = L, K = S.  The second operand is X^T (N x K,
  // K contiguous) on the 128 x 128 kernel, X itself (K x N) under qtr.
  GemmArgs& u = r.upd;
  u.P = static_cast<const char*>(wb.B); u.p_mat = matA; u.ldp = cg.S * es;
  if (qtr) {
    u.Q = X; u.q_mat = matX; u.ldq = cg.L * es;
    u.p_mode = 1;  // B: upper-triangle tiles
    u.q_mode = 2;  // X: K x N
  } else {
    u.Q = XTc; u.q_mat = matX; u.ldq = cg.S * es;
  }
  u.k_slabs = cg.S * es / 128;
  u.tiles_m = ts; u.tiles_n = tl; u.syrk = 0; u.tiles_per_mat = ts * tl;
  u.E = X; u.e_mat = matX; u.lde = cg.L * es;
  u.alpha = a;
  u.s = cg.s; u.l = cg.l;
  u.xscale = k == 0 ? wb.xscale : nullptr;  // X1 = r (a X~ + B0 X~)
  r.f[2] = nm * 2 * s * s * l; r.x[2] = nm * 2 * Sp * Sp * Lp;
  r.last = k + 1 == K;
  if (!r.last) {
    u.C = static_cast<char*>(wb.X[cur ^ 1]); u.c_mat = matX; u.ldc = cg.L * es;
    if (!qtr) { u.CT = static_cast<char*>(wb.XT[cur ^ 1]); u.ct_mat = matX; u.ldct = cg.S * es; }
    // reads B, X (twice under qtr, else X^T and X); writes X' (and X'^T)
    r.b[2] = nm * (s * s + (qtr ? 3 : 4) * s * l) * xsz;
  } else {
    u.desc = d_desc; u.final_kind = sc.final_kind; u.param_dtype = cg.param_dtype;
    // reads B, X^T, X (and W); writes W or out
    r.b[2] = nm * ((s * s + 2 * s * l) * xsz + s * l * (sc.final_kind == 0 ? 2 * psz : psz));
  }
  return r;
}

template <typename GT, typename XT>
hipError_t run_chunk_t(const ChunkGeom& cg, const MatDesc* d_desc, const ChunkBuffers& wb,
                       const StepScalars& sc, const float* coeffs, int K, hipStream_t st,
                       LaunchTimer* timer) {
  if (wb.sync) return run_small<GT, XT>(cg, d_desc, wb, sc, coeffs, K, st, timer);
  hipError_t e = run_prologue_t<GT, XT>(cg, d_desc, wb, sc, coeffs, K, st, timer);
  if (e != hipSuccess || K == 0) return e;
  const bool qtr = !chunk_keeps_xt(cg.S, cg.L, sizeof(XT) == 4, K);
  const int nmat = cg.nmat;
  int cur = 0;
  for (int k = 0; k < K; ++k) {
    const StepProducts sp = step_products<XT>(cg, d_desc, wb, sc, coeffs, K, k, cur);
    {
      Timed tm(timer, KK_GRAM, st);
      if ((e = launch_gemm<XT>(EPI_GRAM, sp.gram, nmat, st)) != hipSuccess) return e;
      tm.done(sp.f[0], sp.x[0], sp.b[0]);
    }
    {
      Timed tm(timer, KK_POLY, st);
      if ((e = launch_gemm<XT>(EPI_POLY, sp.poly, nmat, st)) != hipSuccess) return e;
      tm.done(sp.f[1], sp.x[1], sp.b[1]);
    }
    {
      const int epi = sp.last ? EPI_FINAL : EPI_UPDATE;
      Timed tm(timer, sp.last ? KK_FINAL : KK_UPDATE, st);
      if ((e = qtr ? launch_tile<CfgSquare>(epi, sp.upd, nmat, st) : launch_gemm<XT>(epi, sp.upd, nmat, st)) !=
          hipSuccess)
        return e;
      tm.done(sp.f[2], sp.x[2], sp.b[2]);
    }
    cur ^= 1;
  }
  return hipSuccess;
}

}  // namespace

hipError_t run_chunk(const ChunkGeom& cg, const MatDesc* d_desc, const ChunkBuffers& wb,
                     const StepScalars& sc, const float* coeffs, int K, hipStream_t st,
                     LaunchTimer* timer) {
  const bool gbf = cg.grad_dtype == DT_BF16;
  if (cg.ns_f32) {
    return gbf ? run_chunk_t<uint16_t, float>(cg, d_desc, wb, sc, coeffs, K, st, timer)
               : run_chunk_t<float, float>(cg, d_desc, wb, sc, coeffs, K, st, timer);
  }
  return gbf ? run_chunk_t<uint16_t, uint16_t>(cg, d_desc, wb, sc, coeffs, K, st, timer)
             : run_chunk_t<float, uint16_t>(cg, d_desc, wb, sc, coeffs, K, st, timer);
}

bool group_eligible(const ChunkGeom& cg, int K) {
  return !cg.ns_f32 && K > 0 && cg.S % 256 == 0 && cg.L % 256 == 0 && tile_rows_fit(cg.S, cg.L, 2) &&
         !chunk_is_small(cg.s, cg.l, false);
}

hipError_t run_group(const GroupMember* m, int n, const StepScalars& sc, int K, hipStream_t st,
                     LaunchTimer* timer) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  for (int c = 0; c < n; ++c)
    if (!group_eligible(m[c].geom, K) || m[c].geom.param_dtype != m[0].geom.param_dtype) return hipErrorInvalidValue;
  hipError_t e;
  for (int c = 0; c < n; ++c) {
    const bool gbf = m[c].geom.grad_dtype == DT_BF16;
    e = gbf ? run_prologue_t<uint16_t, uint16_t>(m[c].geom, m[c].desc, m[c].wb, sc, m[c].coeffs, K, st, timer)
            : run_prologue_t<float, uint16_t>(m[c].geom, m[c].desc, m[c].wb, sc, m[c].coeffs, K, st, timer);
    if (e != hipSuccess) return e;
  }
  int cur = 0;
  for (int k = 0; k < K; ++k) {
    GemmArgs ga[3][kMaxGroup];
    int nm[kMaxGroup];
    double f[3] = {0, 0, 0}, x[3] = {0, 0, 0}, b[3] = {0, 0, 0};
    bool last = false;
    for (int c = 0; c < n; ++c) {
      const StepProducts sp = step_products<uint16_t>(m[c].geom, m[c].desc, m[c].wb, sc, m[c].coeffs, K, k, cur);
      ga[0][c] = sp.gram; ga[1][c] = sp.poly; ga[2][c] = sp.upd;
      nm[c] = m[c].geom.nmat;
      for (int q = 0; q < 3; ++q) { f[q] += sp.f[q]; x[q] += sp.x[q]; b[q] += sp.b[q]; }
      last = sp.last;
    }
    const int kinds[3] = {KK_GRAM, KK_POLY, last ? KK_FINAL : KK_UPDATE};
    const int epis[3] = {EPI_GRAM, EPI_POLY, last ? EPI_FINAL : EPI_UPDATE};
    for (int q = 0; q < 3; ++q) {
      Timed tm(timer, kinds[q], st);
      if ((e = launch_group<CfgSquare>(epis[q], ga[q], nm, n, st)) != hipSuccess) return e;
      tm.done(f[q], x[q], b[q]);
    }
    cur ^= 1;
  }
  return hipSuccess;
}

// ---------------------------------------------------------------------------
// AdamW over many tensors in one launch: workgroup b updates elements
// [8192 j, 8192 (j + 1)) of the tensor whose range of workgroups holds b
// (found by binary search over first_block).  HBM-bound: each element reads
// p, g, m, v and writes p, m, v once; 8 consecutive elements per thread
// (16-byte accesses) when the tensor allows it.
// ---------------------------------------------------------------------------
template <typename PT, typename GT>
__device__ __forceinline__ void adam_one(float& p, float g, float& m, float& v, const AdamScalars& sc) {
  m = fmaf(sc.beta1, m, sc.one_minus_beta1 * g);
  v = fmaf(sc.beta2, v, sc.one_minus_beta2 * (g * g));
  const float denom = fmaf(sqrtf(v), sc.inv_sqrt_bc2, sc.eps);
  p = fmaf(p, sc.decay, -sc.step_size * (m / denom));
}

template <typename PT, typename GT>
__global__ __launch_bounds__(256) void k_adamw(const AdamDesc* __restrict__ desc, int n, AdamScalars sc) {
  const int64_t b = blockIdx.x;
  int lo = 0, hi = n - 1;  // last tensor with first_block <= b
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (desc[mid].first_block <= b) lo = mid;
    else hi = mid - 1;
  }
  const AdamDesc a = desc[lo];
  const int64_t start = (b - a.first_block) * kAdamElemsPerBlock;
  const int64_t end = min(a.numel, start + static_cast<int64_t>(kAdamElemsPerBlock));
  PT* __restrict__ p = static_cast<PT*>(a.p);
  const GT* __restrict__ g = static_cast<const GT*>(a.g);
  float* __restrict__ m = a.m;
  float* __restrict__ v = a.v;
  if (a.vec_ok) {
    for (int64_t i = start + threadIdx.x * 8; i < end; i += 256 * 8) {
      float pv[8], gv[8], mv[8], vv[8];
      load8(p, i, pv);
      load8(g, i, gv);
      load8(m, i, mv);
      load8(v, i, vv);
#pragma unroll
      for (int q = 0; q < 8; ++q) adam_one<PT, GT>(pv[q], gv[q], mv[q], vv[q], sc);
      store8(p, i, pv);
      store8(m, i, mv);
      store8(v, i, vv);
    }
  } else {
    for (int64_t i = start + threadIdx.x; i < end; i += 256) {
      float pv = to_f32<PT>(p[i]), mv = m[i], vv = v[i];
      adam_one<PT, GT>(pv, to_f32<GT>(g[i]), mv, vv, sc);
      p[i] = from_f32<PT>(pv);
      m[i] = mv;
      v[i] = vv;
    }
  }
}

// Descriptor records copied into device memory by a kernel that takes them
// as its arguments: the allocation-free entry point fills its table this
// way, with no host staging buffer.  Indices are compile-time constants, so
// the records are read straight from the argument segment.
namespace {
__global__ __launch_bounds__(64) void k_put_desc(DescBatch b, MatDesc* __restrict__ dst) {
  if (threadIdx.x != 0) return;
#pragma unroll
  for (int i = 0; i < kDescPerLaunch; ++i)
    if (i < b.n) dst[i] = b.d[i];
}
}  // namespace

hipError_t put_descriptors(const MatDesc* host, int n, MatDesc* dev, hipStream_t st) {
  for (int first = 0; first < n; first += kDescPerLaunch) {
    DescBatch b{};
    b.n = min(kDescPerLaunch, n - first);
    for (int i = 0; i < b.n; ++i) b.d[i] = host[first + i];
    hipLaunchKernelGGL(k_put_desc, dim3(1), dim3(64), 0, st, b, dev + first);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Streaming copy, the reference for what HBM delivers to the elementwise
// kernels: each workgroup copies its own contiguous 256 KiB with 16-byte
// non-temporal accesses, four in flight per thread (measured the fastest of
// grid-stride and block-contiguous variants, 1-8 accesses per thread).
namespace {
constexpr int64_t kCopyVecsPerBlock = 16384;
__global__ __launch_bounds__(256) void k_stream_copy(const u32x4_t* __restrict__ src, u32x4_t* __restrict__ dst,
                                                     int64_t n) {
  const int64_t lo = static_cast<int64_t>(blockIdx.x) * kCopyVecsPerBlock;
  const int64_t hi = min(lo + kCopyVecsPerBlock, n);
  for (int64_t i = lo + threadIdx.x; i < hi; i += 4 * 256) {
    u32x4_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (i + u * 256 < hi) v[u] = __builtin_nontemporal_load(src + i + u * 256);
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (i + u * 256 < hi) __builtin_nontemporal_store(v[u], dst + i + u * 256);
  }
}
__global__ __launch_bounds__(256) void k_copy_tail(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                                   int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) dst[i] = src[i];
}
}  // namespace

hipError_t stream_copy(void* dst, const void* src, size_t bytes, hipStream_t st) {
  const int64_t vecs = static_cast<int64_t>(bytes / 16);
  if (vecs > 0) {
    const int64_t blocks = (vecs + kCopyVecsPerBlock - 1) / kCopyVecsPerBlock;
    hipLaunchKernelGGL(k_stream_copy, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st,
                       static_cast<const u32x4_t*>(src), static_cast<u32x4_t*>(dst), vecs);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int64_t tail = static_cast<int64_t>(bytes % 16);
  if (tail > 0) {
    hipLaunchKernelGGL(k_copy_tail, dim3(1), dim3(256), 0, st, static_cast<const uint8_t*>(src) + vecs * 16,
                       static_cast<uint8_t*>(dst) + vecs * 16, tail);
    return hipGetLastError();
  }
  return hipSuccess;
}

hipError_t run_adamw(const AdamDesc* d_desc, int n, int64_t blocks, int param_dtype, int grad_dtype,
                     const AdamScalars& sc, double bytes, hipStream_t st, LaunchTimer* timer) {
  if (n <= 0 || blocks <= 0) return hipSuccess;
  Timed tm(timer, KK_ADAMW, st);
  const dim3 grid(static_cast<unsigned>(blocks)), block(256);
  const bool pb = param_dtype == DT_BF16, gb = grad_dtype == DT_BF16;
  if (pb && gb) hipLaunchKernelGGL((k_adamw<uint16_t, uint16_t>), grid, block, 0, st, d_desc, n, sc);
  else if (pb) hipLaunchKernelGGL((k_adamw<uint16_t, float>), grid, block, 0, st, d_desc, n, sc);
  else if (gb) hipLaunchKernelGGL((k_adamw<float, uint16_t>), grid, block, 0, st, d_desc, n, sc);
  else hipLaunchKernelGGL((k_adamw<float, float>), grid, block, 0, st, d_desc, n, sc);
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess) tm.done(0, 0, bytes);
  return e;
}

}  // namespace muon
