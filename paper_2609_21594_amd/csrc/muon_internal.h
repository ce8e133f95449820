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

enum DType : int32_t { DT_F32 = 0, DT_BF16 = 1 };

// One matrix of a chunk, as the kernels see it (device-resident table).
// The matrix is a logical view of the caller's storage: its row i starts at
// element (i / rb) * bstride + (i % rb) * ld of W, g and out, and at
// (i / rb) * bstride_b + (i % rb) * ld_b of buf; the cols elements of a row
// are contiguous.  A dense matrix has ld = cols, rb = rows.
struct MatDesc {
  void* W;              // parameter (muon_step), param dtype
  const void* g;        // gradient (muon_step) or NS input (orthogonalize)
  float* buf;           // momentum (muon_step), fp32
  void* out;            // output (orthogonalize)
  int32_t rows, cols;   // the logical matrix
  int32_t transposed;   // rows > cols: the iteration runs on the transpose
  int32_t vec_ok;       // g and buf can be read 8 elements at a time (16-byte aligned)
  float upd_scale;      // lr * RMS-matching scale
  float decay;          // 1 - lr * weight_decay
  int32_t vec4_ok;      // W (or out) can be accessed 4 elements at a time
  int32_t dense;        // W, g, buf all dense: element (i, j) at i * cols + j
  int64_t ld, bstride;  // row and row-block strides of W, g, out (elements)
  int64_t ld_b, bstride_b;  // the same for buf
  int32_t rb;           // rows per row block (rows when not interleaved)
  int32_t row8_ok;      // every row of g (and buf) starts 16-byte aligned and cols % 8 == 0
  int32_t reserved[2];
};
static_assert(sizeof(MatDesc) == 112, "MatDesc layout");

// Element offset of row i, column j of the view (W, g, out) and of buf.
__host__ __device__ inline int64_t view_index(const MatDesc& d, int64_t i, int64_t j) {
  if (d.rb >= d.rows) return i * d.ld + j;
  const int64_t q = i / d.rb;
  return q * d.bstride + (i - q * d.rb) * d.ld + j;
}
__host__ __device__ inline int64_t buf_index(const MatDesc& d, int64_t i, int64_t j) {
  if (d.rb >= d.rows) return i * d.ld_b + j;
  const int64_t q = i / d.rb;
  return q * d.bstride_b + (i - q * d.rb) * d.ld_b + j;
}

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
  double* partials;     // nmat x norm_tiles(S, L) (at least kSmallMaxGroup), sums of u^2 in fp64
  unsigned* sync;       // group counters of the fused small-matrix launch (chunk_is_small), or null
  double* rscale;       // nmat: r = 1 / (||u||_F + eps), fp64
  float* xscale;        // nmat: the scale the first Newton-Schulz step applies
                        // to X: r, or 1 where X already holds r*u
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
  KK_APPLY_X0, KK_ADAMW, KK_SMALL, KK_COUNT
};

// Receives a bracket around every launch when timing is enabled.
struct LaunchTimer {
  virtual void begin(int kind, hipStream_t st) = 0;
  virtual void end(int kind, hipStream_t st, double flops, double exec_flops, double bytes) = 0;
  virtual ~LaunchTimer() = default;
};

inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }
// Norm partial sums per matrix: one per 64x64 tile of the padded extent.
inline int64_t norm_tiles(int64_t S, int64_t L) { return (S / 64) * (L / 64); }

// The 256 x 256 kernel addresses a tile's 256 rows (operands, the a*X
// term, the parameter block) by 32-bit offsets from one base, so every row
// it reads or writes must be shorter than 2^31 / 256 bytes.
constexpr int64_t kTileMaxRowBytes = (int64_t(1) << 31) / 256;
inline bool tile_rows_fit(int64_t S, int64_t L, int es) {
  return S * es < kTileMaxRowBytes && L * es < kTileMaxRowBytes;
}
// A chunk keeps X^T (two more X-sized workspace buffers) unless its update
// products run on the 256 x 256 kernel, which reads X itself through
// transposing LDS reads: bf16 Newton-Schulz, S and L multiples of 256, at
// least one step, rows within that kernel's offsets.
inline bool chunk_keeps_xt(int64_t S, int64_t L, bool ns_f32, int K) {
  return ns_f32 || S % 256 != 0 || L % 256 != 0 || K == 0 || !tile_rows_fit(S, L, 2);
}
// A chunk runs as one fused launch (k_ns_small: momentum, norm, every
// Newton-Schulz step and the update) when its short side is at most 128 and
// the fused launch is the faster one for its shape: always for fp32 NS; for
// bf16 NS when the short side is at most 64 or the long side at most 512
// (measured: 64 matrices of 128 x 2048 run twice as fast as 128 x 128 tiles,
// whose operand units carry four times the flops per byte).  The choice
// depends on the shape alone, so a matrix gets the same bits in any batch.
// Such a chunk also needs the group counters (kSmallSyncBytes) and
// kSmallMaxGroup norm partials per matrix.
constexpr int kSmallMaxGroup = 32;
constexpr int64_t kSmallSyncBytes = 64 * 1024;
inline bool chunk_is_small(int64_t s, int64_t l, bool ns_f32) {
  if (s > 128 || l > (int64_t(1) << 16)) return false;
  return ns_f32 || s <= 64 || l <= 512;
}

// A group: chunks whose products of each Newton-Schulz step run as one
// launch per product (the 256 x 256 kernel over all their tiles).  Each
// member has its own workspace; they share the step count, the NS precision
// (bf16) and the parameter dtype.
struct GroupMember {
  ChunkGeom geom;
  const MatDesc* desc;
  ChunkBuffers wb;
  const float* coeffs;  // host, K x 3
};
constexpr int kGroupMax = 8;
// A chunk can join a group: bf16 NS on the 256 x 256 kernels (padded
// extents multiples of 256, rows within its offsets), at least one step,
// not a fused small-matrix chunk.
bool group_eligible(const ChunkGeom& g, int K);
hipError_t run_group(const GroupMember* members, int n, const StepScalars& sc, int K, hipStream_t stream,
                     LaunchTimer* timer);

// ---------------------------------------------------------------------------
// AdamW for the parameters Muon does not take (1-D and scalar ones; Sec. 6.4
// delegates them to AdamW through a chained optimizer).
// ---------------------------------------------------------------------------
// Elements one workgroup updates.
constexpr int kAdamElemsPerBlock = 8192;

// One tensor of an AdamW call (device-resident table).
struct AdamDesc {
  void* p;              // parameter, param dtype
  const void* g;        // gradient, grad dtype
  float* m;             // first moment, fp32
  float* v;             // second moment, fp32
  int64_t numel;
  int64_t first_block;  // workgroups of the launch before this tensor's
  int32_t vec_ok;       // 8 elements at a time: numel % 8 == 0 and 16-byte aligned
  int32_t reserved[3];
};
static_assert(sizeof(AdamDesc) == 64, "AdamDesc layout");

// Per-call scalars: p' = p*decay - step_size * m' / (sqrt(v')*inv_sqrt_bc2 + eps),
// m' = beta1*m + (1-beta1)*g, v' = beta2*v + (1-beta2)*g^2.
struct AdamScalars {
  float decay;          // 1 - lr*wd
  float beta1, one_minus_beta1, beta2, one_minus_beta2;
  float step_size;      // lr / (1 - beta1^t)
  float inv_sqrt_bc2;   // 1 / sqrt(1 - beta2^t)
  float eps;
};

// Updates n tensors of one (param, grad) dtype pair: `blocks` workgroups.
hipError_t run_adamw(const AdamDesc* d_desc, int n, int64_t blocks, int param_dtype,
                     int grad_dtype, const AdamScalars& sc, double bytes, hipStream_t stream,
                     LaunchTimer* timer);

// Copies n descriptor records from host memory into the device table `dev`
// on `stream`, as kernel arguments (kDescPerLaunch records per launch): no
// staging buffer and no allocation.
constexpr int kDescPerLaunch = 16;
struct DescBatch {
  int32_t n;
  int32_t pad[3];
  MatDesc d[kDescPerLaunch];
};
hipError_t put_descriptors(const MatDesc* host, int n, MatDesc* dev, hipStream_t stream);

// The HBM reference copy (dst and src 16-byte aligned, not overlapping).
hipError_t stream_copy(void* dst, const void* src, size_t bytes, hipStream_t stream);

// Enqueues the whole step for one chunk on `stream`: momentum + partial
// norms, norm finalisation, normalise + transpose-first + cast, K
// Newton-Schulz steps (Gram, polynomial, update), and the final apply.
hipError_t run_chunk(const ChunkGeom& g, const MatDesc* d_desc, const ChunkBuffers& wb,
                     const StepScalars& sc, const float* coeffs /* host, K x 3 */, int K,
                     hipStream_t stream, LaunchTimer* timer /* may be null */);

}  // namespace muon
