// CPU check of the SYRK planner's arithmetic (host-only header): for row
// strides up to the accepted maximum, every K-slice spans at most 2^31 bytes
// (descriptor ranges and stage offsets are 32-bit), the chunks cover the
// rows, and the workspace query (no stride limit) is large enough for every
// stride's plan; and for the slices at the end of every chunk, the last
// stage that holds rows starts inside the slice's descriptor range (the
// per-stage descriptor advance subtracts the stage offset from the range
// without clamping).  Prints "ok" or the first violation and exits non-zero.
#include <cstdio>
#include <cstdlib>

#include "syrk_plan.h"

int main() {
  const long long rows[] = {1, 63, 64, 1000, 8191, 8192, 16383, 16384, 21900, 24575, 65536,
                            100000, 131072, 200000, 262144, 262145, 300000, 500000, 523264,
                            524288, 524289, 600000, 1000000, 1048576, 4000000, 10000000};
  const long long Ds[] = {64, 320, 2048, 4096, 8192, 32768};
  const long long lds[] = {0, 64, 8192, 16384, 20000, 32768, 32832, 40000, 50000, 65536};
  long long checked = 0;
  for (long long n : rows)
    for (long long D : Ds)
      for (long long ldx : lds) {
        if (ldx && ldx < D) continue;
        const attr::SyrkPlan P = attr::plan_syrk(n, D, ldx);
        const attr::SyrkPlan Q = attr::plan_syrk(n, D, 0);
        const long long ld = ldx ? ldx : D;
        const long long n_chunks = (n + P.C - 1) / P.C;
        bool ok = P.J >= 1 && P.J <= attr::kSyrkSlices && (P.J == 1 || P.J % 2 == 0) &&
                  P.Cs % 64 == 0 && P.Cs >= 64 &&
                  P.C == P.Cs * P.J && n_chunks * P.C >= n && P.part_bytes <= Q.part_bytes &&
                  P.h64_bytes == Q.h64_bytes;
        if (ldx) ok = ok && P.Cs * ld * 2 <= (1ll << 31);
        // the kernel's slice range (bytes from the tile's first column) for
        // the first and the last column tile, at the first and the last
        // slice of every chunk (plans that launch: a given stride)
        for (long long r0 = 0; ok && ldx && r0 < n; r0 += P.C) {
          const long long rows_c = n - r0 < P.C ? n - r0 : P.C;
          const long long Jc = (rows_c + P.Cs - 1) / P.Cs;
          for (long long j : {0ll, Jc - 1}) {
            const long long rs = r0 + j * P.Cs;
            long long nr = n - rs;
            nr = nr > P.Cs ? P.Cs : nr;
            if (nr <= 0) continue;
            const long long n_st = (nr + 63) / 64;
            for (long long c0 : {0ll, (D - 1) / 256 * 256}) {
              const long long lim_slice = nr * ld, lim_mat = (n - 1 - rs) * ld + (D - c0);
              const long long range = 2 * (lim_slice < lim_mat ? lim_slice : lim_mat);
              const long long off = (n_st - 1) * 64 * ld * 2;
              ok = ok && off < range && range < (1ll << 32);
            }
          }
        }
        if (!ok) {
          std::printf("violation: n=%lld D=%lld ldx=%lld -> J=%d Cs=%lld C=%lld part=%zu (query %zu)\n",
                      n, D, ldx, P.J, (long long)P.Cs, (long long)P.C, P.part_bytes, Q.part_bytes);
          return 1;
        }
        ++checked;
      }
  // the case that used to wrap: a full 524288-row chunk at the largest stride
  const attr::SyrkPlan W = attr::plan_syrk(524288, 8192, 65536);
  if (W.Cs * 65536ll * 2 > (1ll << 31)) {
    std::printf("violation: 524288 rows at ldx 65536 give %lld-row slices\n", (long long)W.Cs);
    return 1;
  }
  // the cost model's choices on the workloads it was tuned for: 10^6 x 8192
  // (two chunks of 16 slices of 31296 rows), K-FAC factors over 21900 rows
  const attr::SyrkPlan A = attr::plan_syrk(1000000, 8192, 8192);
  const attr::SyrkPlan B = attr::plan_syrk(21900, 2048, 2048);
  const attr::SyrkPlan C = attr::plan_syrk(21900, 8192, 8192);
  if (A.J != 16 || A.Cs != 31296 || B.J != 6 || C.J != 4) {
    std::printf("unexpected plans: 10^6x8192 J=%d Cs=%lld, 21900x2048 J=%d, 21900x8192 J=%d\n", A.J,
                (long long)A.Cs, B.J, C.J);
    return 1;
  }
  std::printf("ok %lld plans\n", checked);
  return 0;
}
