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

// Rows of one K-slice must span at most 2^31 bytes: the GEMM core's buffer
// descriptor range, its per-lane offsets and its per-stage descriptor
// advance are 32-bit quantities.
inline int64_t syrk_max_slice_rows(int64_t ldx) {
  if (ldx <= 0) return INT64_MAX;
  int64_t r = ((int64_t)1 << 30) / ldx;  // rows of 2 * ldx bytes in 2^31 bytes
  return r / 64 * 64;
}

// Equal chunks of at most max_chunk rows (10^6 rows: two of 500000 rather
// than one full chunk and a ragged one), rounded up to 64-row stages.
inline int64_t syrk_chunk_rows(int64_t n_rows, int64_t max_chunk) {
  const int64_t n_chunks = n_rows > max_chunk ? (n_rows + max_chunk - 1) / max_chunk : 1;
  int64_t c = (n_rows + n_chunks - 1) / n_chunks;
  c = (c + 63) / 64 * 64;
  return c < 64 ? 64 : c;
}

// K-slices of a chunk of c rows: the count (1 or even, so that the slices of
// either sign pair up; at least Jmin; at most kSyrkSlices; no empty slice)
// with the least modelled time: whole rounds of 256 workgroups (one per CU:
// the GEMM core takes 128 KB of LDS) times the 64-row stages of a slice
// plus ~12 stage-times for the partial tile each slice writes and the
// reduction reads back.  Ties go to fewer slices.  10^6 x 8192: 16 slices of
// 31296 rows (33 whole rounds); 21900 token rows at D = 2048 (36 tiles): 6
// slices in one round instead of 15 in three; at D = 8192: 4 slices.
inline int syrk_slices(int64_t c, int n_up, int Jmin) {
  int best = 0;
  int64_t best_cost = INT64_MAX;
  for (int J = 1; J <= kSyrkSlices; J = J == 1 ? 2 : J + 2) {
    if (J < Jmin) continue;
    int64_t cs = (c + J - 1) / J;
    cs = (cs + 63) / 64 * 64;
    if (J > 1 && (int64_t)(J - 1) * cs >= c && best > 0) break;  // an empty last slice
    const int64_t rounds = ((int64_t)J * n_up + 255) / 256;
    const int64_t cost = rounds * (cs / 64 + 12);
    if (cost < best_cost) {
      best_cost = cost;
      best = J;
    }
  }
  return best;
}

// ldx: row stride of X in elements, or 0 for the workspace query.  The
// query's plan (no stride limit) fixes the slice count Jq and with it the
// partial-tile workspace; a stride whose slices would then exceed
// syrk_max_slice_rows(ldx) rows takes shorter chunks (at most Jq such slices
// each) and never more than Jq slices, so the query covers every stride.
inline SyrkPlan plan_syrk(int64_t n_rows, int64_t D, int64_t ldx) {
  SyrkPlan P{};
  P.nt = (int)((D + kSyrkTile - 1) / kSyrkTile);
  P.n_up = P.nt * (P.nt + 1) / 2;
  int64_t c = syrk_chunk_rows(n_rows, kSyrkChunkRows);
  const int Jq = syrk_slices(c, P.n_up, 1);
  int J = Jq;
  const int64_t max_cs = syrk_max_slice_rows(ldx);
  if (ldx > 0 && ((c + Jq - 1) / Jq + 63) / 64 * 64 > max_cs) {
    const int64_t lim = max_cs * Jq;
    c = syrk_chunk_rows(n_rows, lim < kSyrkChunkRows ? lim : kSyrkChunkRows);
    int Jmin = (int)((c + max_cs - 1) / max_cs);  // <= Jq (c <= Jq max_cs)
    if (Jmin > 1 && (Jmin & 1)) ++Jmin;           // Jq is 1 or even
    J = syrk_slices(c, P.n_up, Jmin);
    if (J > Jq) J = Jq;
  }
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
