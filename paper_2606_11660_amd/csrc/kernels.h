// Internal interface between the C-ABI layer (api.cpp) and the HIP kernels.
// Nothing here is exported from the shared library.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace attr {

// ---------------------------------------------------------------------------
// projection
// ---------------------------------------------------------------------------
// One module slot of the projection's device-side table (slots are in
// launch order, largest modules first).
struct ProjTab {
  const void* a;
  const void* g;
  const void* pk;     // packed S fragments, then packed R fragments
  int64_t lda, ldg, out_col;
  int32_t d_in, d_out;
};

// One work group of the projection: ms consecutive slots from slot0 whose
// modules share their input rows (ms = 1 for a module on its own).
struct ProjGroup {
  int32_t slot0, ms;
};

// Host -> device upload of module descriptors travels in kernel arguments.
struct PackEntry {
  const void* a;
  const void* g;
  const void* R;
  const void* S;
  const float* v_out;  // optional factored second moment (both or neither)
  const float* v_in;
  int64_t lda, ldg, out_col, pk_off;
  int32_t d_in, d_out;
  int32_t grp;      // group of this slot
  int32_t lead_ms;  // group size if this slot is the group's first, else 0
};
constexpr int kPackMax = 24;
struct PackArgs {
  PackEntry e[kPackMax];
  int32_t n;
  int32_t slot0;
};

// Tokens handled by one workgroup of the projection for fragment width nk
// (k = 16 * nk).
int project_chunk_tokens(int nk);
// Bytes of packed S and R for one module.
size_t project_packed_bytes(int64_t d_in, int64_t d_out, int k, int elem_bytes);

// Static device scratch of attr_project_noalloc (per GPU, 256-byte aligned):
// its device address on the current device, resolved once per device.
constexpr size_t kProjectScratchBytes = (size_t)64 << 20;
hipError_t project_scratch(void** ptr);

hipError_t launch_project_pack(bool bf16, int nk, const PackArgs& args, ProjTab* tab,
                               ProjGroup* gtab, char* pk_base, hipStream_t s);
// Modules sharing their input rows (same a, lda, d_in) are projected in
// groups of up to kProjGroupMax consecutive slots (one read of a per group).
// One launch covers every (group, token chunk, example) item, groups in
// table order (largest work first).
constexpr int kProjGroupMax = 3;
// Work list of a call with per-example lengths (device-built): examples
// sorted by chunk count, longest first, and the item offset of each chunk
// row.  Built when length is given, n_chunks <= kWorklistMaxChunks and
// n_examples <= kWorklistMaxExamples; otherwise the main kernel decodes its
// block index densely.
constexpr int kWorklistMaxChunks = 2048;
constexpr int64_t kWorklistMaxExamples = 1 << 20;
inline bool project_uses_worklist(const int32_t* length, int64_t n_ex, int n_chunks) {
  return length && n_chunks <= kWorklistMaxChunks && n_ex <= kWorklistMaxExamples;
}
// tok: per-token blocks written straight into `partial` = the output [n_rows, ldo]
// wl_perm / wl_off: the work list (both NULL for the dense decode).
hipError_t launch_project_main(bool bf16, int nk, const ProjTab* tab, const ProjGroup* gtab,
                               int n_groups, int n_chunks, int64_t n_ex, int64_t T,
                               const int64_t* row_offset, const int32_t* length,
                               int32_t* wl_perm, int32_t* wl_off,
                               float* partial, hipStream_t s, bool tok = false, int64_t ldo = 0,
                               int64_t n_rows = 0);
hipError_t launch_project_reduce(int nk, const ProjTab* tab, int n_slots, int n_chunks,
                                 int64_t n_ex, int64_t T, const int32_t* length,
                                 const float* partial, float* out, int64_t ldo,
                                 hipStream_t s);

// ---------------------------------------------------------------------------
// row-wise preconditioning / normalisation (NONE and DIAG)
// ---------------------------------------------------------------------------
// x_dtype / y_dtype: 0 = fp32, 2 = fp16 (attr_dtype values).
// row_ss (optional): n_ss partial sums of squares per row that give the
// norm; seg_e (optional, with row_ss): per row, the exponent e of each
// 128-column segment of X, which holds y 2^-e (y = X 2^e is normalised).
hipError_t launch_rowscale(int x_dtype, int y_dtype, const void* X, int64_t ldx,
                           int64_t n_rows, int64_t D, const float* m, int unit,
                           const float* row_ss, const int8_t* seg_e, int64_t n_ss, void* Y,
                           int64_t ldy, hipStream_t s);

// ---------------------------------------------------------------------------
// diagonal accumulate
// ---------------------------------------------------------------------------
int colsumsq_panels(int64_t n_rows, int64_t D);
hipError_t launch_colsumsq(int x_dtype, const void* X, int64_t ldx, int64_t n_rows,
                           int64_t D, float* H, double* part, hipStream_t s);

// ---------------------------------------------------------------------------
// scoring
// ---------------------------------------------------------------------------
struct ScorePlan {
  int n_qb;              // query blocks of 64 queries
  int n_grp;             // 128-byte K-groups per row
  int split;             // D-slices (1: fused plan)
  int n_tiles;           // 128-row tiles (split-K plan)
  int n_parts;           // row partitions, one sorted list each per query
  int64_t rows_per_part;
  size_t spart_bytes;    // split-K partial scores / GEMM-plan score chunk
  size_t list_entries;   // n_q * n_parts * k
  int gemm;              // GEMM plan (1: 256 x 256 tiles, 2: 128 x 256 ring): row chunks of `chunk` rows, one list per chunk
  int64_t chunk;
  int64_t D;
  int64_t bound_rows;    // streaming plan: rows of the prefix scan that bounds the k-th best (0: none)
};
ScorePlan plan_score(int64_t n_q, int64_t n_g, int64_t D, int k, int elem_bytes);
hipError_t launch_score_topk(bool f16, const ScorePlan& plan, const void* Q, int64_t n_q,
                             int64_t ldq, const void* G, int64_t n_g, int64_t ldg, int k,
                             int64_t index_base, int merge, float* top_s, int64_t* top_i,
                             float* part_s, int64_t* part_i, float* spart, hipStream_t s);

// ---------------------------------------------------------------------------
// full second moment: accumulate (SYRK) and apply
// ---------------------------------------------------------------------------
struct SyrkPlan {
  int nt;          // 256-wide tiles per side
  int n_up;        // upper-triangle tiles
  int J;           // K-slices per chunk
  int64_t Cs;      // rows per slice
  int64_t C;       // rows per chunk (J * Cs)
  size_t part_bytes, h64_bytes;
};
// plan_syrk(n_rows, D, ldx) is in syrk_plan.h (host only).
hipError_t launch_syrk(bool bf16, const void* X, int64_t ldx, int64_t n_rows, int64_t D, float* H,
                       const SyrkPlan& P, void* part, void* h64, hipStream_t s);

int apply_full_nss(int64_t D);
size_t apply_full_workspace(int64_t n_rows, int64_t D, int unit);
hipError_t launch_apply_full(const void* X, int64_t n_rows, int64_t ldx, int64_t D, const float* M,
                             int y_dtype, void* Y, int64_t ldy, int unit, void* ws,
                             hipStream_t s);

// ---------------------------------------------------------------------------
// calibration
// ---------------------------------------------------------------------------
hipError_t launch_probe_read(const void* x, size_t bytes, void* sink, hipStream_t s);
hipError_t launch_probe_mfma(int64_t n_mfma, void* sink, hipStream_t s);

}  // namespace attr
