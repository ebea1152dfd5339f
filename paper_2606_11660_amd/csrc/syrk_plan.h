// Host-side plan of the full second-moment accumulation (H += X^T X): row
// chunks per launch, K-slices per chunk and workspace sizes.  Plain C++ with
// no device code, so the arithmetic can be checked on the CPU.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "kernels.h"

namespace attr {

#ifndef ATTR_SYRK_SLICE_ROWS
#define ATTR_SYRK_SLICE_ROWS 32768
#endif
constexpr int kSyrkTile = 256;          // block tile of the GEMM core (both sides)
constexpr int kSyrkSlices = 16;         // K-slices per full chunk (whole rounds of 256 CUs)
constexpr int kSyrkSliceRows = ATTR_SYRK_SLICE_ROWS;        // longest fp32 accumulation
constexpr int kSyrkChunkRows = kSyrkSlices * kSyrkSliceRows;  // rows per launch

// Rows of one K-slice must span at most 2^31 bytes: the GEMM core marks its
// loads past the last stage by adding 2^31 to their offset, which lands out
// of the slice's buffer range only when that range is at most 2^31 bytes.
inline int64_t syrk_max_slice_rows(int64_t ldx) {
  if (ldx <= 0) return INT64_MAX;
  int64_t r = ((int64_t)1 << 30) / ldx;  // rows of 2 * ldx bytes in 2^31 bytes
  return r / 64 * 64;
}

// ldx: row stride of X in elements, or 0 for the workspace query (no stride
// limit: that plan needs at least as much workspace as any stride's plan,
// because a stride limit only shortens chunks, and slices per chunk never
// grow as chunks shrink).
inline SyrkPlan plan_syrk(int64_t n_rows, int64_t D, int64_t ldx) {
  SyrkPlan P{};
  P.nt = (int)((D + kSyrkTile - 1) / kSyrkTile);
  P.n_up = P.nt * (P.nt + 1) / 2;
  int64_t max_chunk = kSyrkChunkRows;
  const int64_t max_cs = syrk_max_slice_rows(ldx);
  if (max_cs < max_chunk / kSyrkSlices) max_chunk = max_cs * kSyrkSlices;
  // equal chunks of at most max_chunk rows (10^6 rows: two of 500000, each
  // 16 slices of 31296, rather than one full chunk and a ragged one)
  const int64_t n_chunks = n_rows > max_chunk ? (n_rows + max_chunk - 1) / max_chunk : 1;
  int64_t c = (n_rows + n_chunks - 1) / n_chunks;
  c = (c + 63) / 64 * 64;
  if (c < 64) c = 64;
  // 16 K-slices, fewer for short chunks (slices of >= 8192 rows: each slice
  // adds a partial tile to write and reduce), but enough for two workgroups
  // per CU when the matrix has few tiles (D = 2048: 36 tiles), with slices
  // of >= 1024 rows
  int J = (int)(c / 8192);
  const int fill = (512 + P.n_up - 1) / P.n_up;
  const int Jmax_short = (int)(c / 1024);
  if (J < fill) J = fill < Jmax_short ? fill : Jmax_short;
  J = J < 1 ? 1 : (J > kSyrkSlices ? kSyrkSlices : J);
  int64_t cs = (c + J - 1) / J;
  cs = (cs + 63) / 64 * 64;
  P.J = J;
  P.Cs = cs;
  P.C = cs * J;
  P.part_bytes = (size_t)J * (size_t)P.n_up * kSyrkTile * kSyrkTile * 4;
  P.h64_bytes = (size_t)P.n_up * kSyrkTile * kSyrkTile * 8;
  return P;
}

}  // namespace attr
