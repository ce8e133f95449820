// Internal interface between the C ABI layer (muon_api.hip) and the gfx950
// kernels (muon_kernels.hip).  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace muon {

// Workspace extents of every matrix are rounded up to this multiple, and the
// padding is kept at zero, so the contraction kernels never test bounds.
constexpr int kPad = 128;
// GEMM macro tile (rows and columns of one workgroup's output tile).
constexpr int kTile = 128;
// Elements reduced by one workgroup of the momentum / norm kernel.
constexpr int kNormElemsPerBlock = 16384;

enum DType : int32_t { DT_F32 = 0, DT_BF16 = 1 };

// One matrix of a chunk, as the kernels see it (device-resident table).
struct MatDesc {
  void* W;              // parameter (muon_step), param dtype, rows x cols
  const void* g;        // gradient (muon_step) or NS input (orthogonalize)
  float* buf;           // momentum (muon_step), fp32
  void* out;            // output (orthogonalize), rows x cols
  int32_t rows, cols;   // the matrix as stored by the caller
  int32_t transposed;   // rows > cols: the iteration runs on the transpose
  int32_t vec_ok;       // 16-byte aligned pointers and rows*cols % 8 == 0
  float upd_scale;      // lr * RMS-matching scale
  float decay;          // 1 - lr * weight_decay
  int32_t vec4_ok;      // W (or out) 16-byte aligned and cols % 4 == 0
  int32_t reserved1;
};
static_assert(sizeof(MatDesc) == 64, "MatDesc layout");

// Geometry shared by all matrices of a chunk.
struct ChunkGeom {
  int32_t s, l;         // short and long side
  int32_t S, L;         // padded extents (multiples of kPad)
  int32_t nmat;
  int32_t ns_f32;       // 1: fp32 NS arithmetic, 0: bf16 operands
  int32_t grad_dtype;   // DType of desc.g
  int32_t param_dtype;  // DType of desc.W / desc.out
};

// Chunk workspace: four X buffers (X, X^T and their successors), A, B, and
// the norm scratch.  Element size is 2 (bf16) or 4 (fp32).
struct ChunkBuffers {
  void* X[2];           // S x L, row stride L
  void* XT[2];          // L x S, row stride S
  void* A;              // S x S
  void* B;              // S x S
  float* partials;      // nmat x nblk
  float* rscale;        // nmat: 1 / (||u||_F + eps)
};

struct StepScalars {
  float beta, one_minus_beta;
  int32_t nesterov;
  int32_t momentum;     // 1: muon_step, 0: orthogonalize only
  float eps;
  int32_t final_kind;   // 0: update W, 1: write out
};

// Kernel families, for the optional per-launch timing.
enum KernelKind : int {
  KK_PARTIALS = 0, KK_FINALIZE, KK_NORMALIZE, KK_GRAM, KK_POLY, KK_UPDATE, KK_FINAL,
  KK_APPLY_X0, KK_COUNT
};

// Receives a bracket around every launch when timing is enabled.
struct LaunchTimer {
  virtual void begin(int kind, hipStream_t st) = 0;
  virtual void end(int kind, hipStream_t st, double flops, double exec_flops, double bytes) = 0;
  virtual ~LaunchTimer() = default;
};

inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }
inline int64_t norm_blocks(int64_t numel) {
  return (numel + kNormElemsPerBlock - 1) / kNormElemsPerBlock;
}

// Enqueues the whole step for one chunk on `stream`: momentum + partial
// norms, norm finalisation, normalise + transpose-first + cast, K
// Newton-Schulz steps (Gram, polynomial, update), and the final apply.
hipError_t run_chunk(const ChunkGeom& g, const MatDesc* d_desc, const ChunkBuffers& wb,
                     const StepScalars& sc, const float* coeffs /* host, K x 3 */, int K,
                     hipStream_t stream, LaunchTimer* timer /* may be null */);

}  // namespace muon
