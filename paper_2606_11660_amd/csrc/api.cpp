// C-ABI layer of libattr: argument validation, workspace layout and kernel
// dispatch.  Every check runs on the host before anything is enqueued, so a
// rejected call leaves all outputs untouched.  See include/attr.h for the
// contract of each entry point.
#include "attr.h"

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <exception>
#include <numeric>
#include <string>
#include <map>
#include <tuple>
#include <vector>

#include "kernels.h"
#include "syrk_plan.h"

namespace {

thread_local std::string g_err;

attr_status fail(attr_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

attr_status device_fail(hipError_t e, const char* what) {
  return fail(ATTR_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

int dtype_bytes(attr_dtype d) { return d == ATTR_F32 ? 4 : 2; }

bool valid_dtype(attr_dtype d) { return d == ATTR_F32 || d == ATTR_BF16 || d == ATTR_F16; }

// Byte range [lo, hi) spanned by a row-major [rows, width] matrix with stride ld.
struct Span {
  uintptr_t lo, hi;
};
Span span_of(const void* p, int64_t rows, int64_t width, int64_t ld, int eb) {
  uintptr_t lo = reinterpret_cast<uintptr_t>(p);
  if (rows <= 0 || width <= 0) return {lo, lo};
  return {lo, lo + (uintptr_t)(((rows - 1) * ld + width) * eb)};
}
bool overlap(Span a, Span b) { return a.lo < b.hi && b.lo < a.hi; }

// ---------------------------------------------------------------------------
// projection
// ---------------------------------------------------------------------------
struct ProjLayout {
  size_t off_tab, off_gtab, off_wl, off_pk, off_part, total;
  std::vector<int> order;       // slot -> module index
  std::vector<size_t> pk_off;   // per slot, relative to off_pk
  std::vector<int> slot_grp;    // slot -> group
  std::vector<int> lead_ms;     // slot -> group size if the group's first slot, else 0
  int n_groups;
  int n_chunks;
};

ProjLayout project_layout(const attr_module* mods, int32_t n_mods, int eb, int64_t n_ex,
                          int64_t T, int k, bool tok = false) {
  ProjLayout L;
  const int nk = k / 16;
  // Modules that read the same input rows (same a, lda and d_in: q/k/v or
  // gate/up of a transformer layer) form groups of up to kProjGroupMax,
  // projected together so that a is read once.  Groups are ordered by their
  // work per token (the row elements they read), largest first, so that the
  // one main launch starts the longest items first and ends on the
  // shortest; a group's members take consecutive slots.
  // (three members at k = 64 would need more than 256 VGPRs: two waves per
  // SIMD no longer fit, so groups stop at two there)
  // (per-token blocks keep one module per item: their row-writing code would
  // pass 256 VGPRs with two or three)
  const size_t gmax = tok ? 1 : (nk >= 4 ? 2 : (size_t)attr::kProjGroupMax);
  std::vector<std::vector<int>> groups;
  std::map<std::tuple<const void*, int64_t, int64_t>, size_t> open;
  for (int x = 0; x < n_mods; ++x) {
    const auto key = std::make_tuple(mods[x].a, (int64_t)mods[x].lda, (int64_t)mods[x].d_in);
    auto it = open.find(key);
    if (it != open.end() && groups[it->second].size() < gmax) {
      groups[it->second].push_back(x);
    } else {
      open[key] = groups.size();
      groups.push_back({x});
    }
  }
  auto cost = [&](const std::vector<int>& gm) {
    int64_t c = mods[gm[0]].d_in;
    for (int x : gm) c += mods[x].d_out;
    return c;
  };
  std::stable_sort(groups.begin(), groups.end(),
                   [&](const std::vector<int>& x, const std::vector<int>& y) {
                     return cost(x) > cost(y);
                   });
  L.n_groups = (int)groups.size();
  for (int gi = 0; gi < L.n_groups; ++gi) {
    const auto& gm = groups[gi];
    for (size_t u = 0; u < gm.size(); ++u) {
      L.order.push_back(gm[u]);
      L.slot_grp.push_back(gi);
      L.lead_ms.push_back(u == 0 ? (int)gm.size() : 0);
    }
  }
  const int CT = attr::project_chunk_tokens(nk);
  L.n_chunks = (int)((T + CT - 1) / CT);
  L.off_tab = 0;
  size_t off = align_up(sizeof(attr::ProjTab) * (size_t)n_mods);
  L.off_gtab = off;
  off += align_up(sizeof(attr::ProjGroup) * (size_t)L.n_groups);
  // work list (examples by chunk count, chunk-row offsets), whether or not
  // the call passes lengths: the query has no lengths to look at
  L.off_wl = off;
  if (n_ex <= attr::kWorklistMaxExamples && L.n_chunks <= attr::kWorklistMaxChunks)
    off += align_up(4 * (size_t)n_ex) + align_up(4 * ((size_t)L.n_chunks + 1));
  L.off_pk = off;
  size_t pk = 0;
  L.pk_off.resize(n_mods);
  for (int sl = 0; sl < n_mods; ++sl) {
    const attr_module& m = mods[L.order[sl]];
    L.pk_off[sl] = pk;
    pk += align_up(attr::project_packed_bytes(m.d_in, m.d_out, k, eb));
  }
  off += pk;
  L.off_part = off;
  off += align_up((size_t)n_mods * (size_t)L.n_chunks * (size_t)n_ex * (size_t)k * k * 4);
  L.total = off;
  return L;
}

attr_status project_validate(const attr_module* mods, int32_t n_mods, attr_dtype in_dtype,
                             int32_t k, int64_t n_ex, int64_t T, float* out, int64_t ldo) {
  if (n_mods < 1 || n_mods > 4096) return fail(ATTR_ERR_INVALID_ARG, "n_mods=%d must be in [1, 4096]", n_mods);
  if (!mods) return fail(ATTR_ERR_INVALID_ARG, "mods is NULL");
  if (in_dtype != ATTR_BF16 && in_dtype != ATTR_F32)
    return fail(ATTR_ERR_UNSUPPORTED, "attr_project: in_dtype must be ATTR_BF16 or ATTR_F32");
  if (k != 16 && k != 32 && k != 64) return fail(ATTR_ERR_UNSUPPORTED, "k=%d must be 16, 32 or 64", k);
  if (n_ex < 0) return fail(ATTR_ERR_INVALID_ARG, "n_examples=%lld is negative", (long long)n_ex);
  if (T < 1) return fail(ATTR_ERR_INVALID_ARG, "T=%lld must be >= 1", (long long)T);
  if (T > (1ll << 24)) return fail(ATTR_ERR_UNSUPPORTED, "T=%lld exceeds 2^24", (long long)T);
  if (n_ex > 0 && !out) return fail(ATTR_ERR_INVALID_ARG, "out is NULL");
  if (!aligned16(out)) return fail(ATTR_ERR_ALIGNMENT, "out must be 16-byte aligned");
  const int eb = dtype_bytes(in_dtype);
  // Rows are streamed in 128-byte groups: 64 bf16 or 32 fp32 values.
  const int KS = in_dtype == ATTR_BF16 ? 64 : 32;
  const int ld_mult = 16 / eb;
  const int64_t kk = (int64_t)k * k;
  if (ldo < kk) return fail(ATTR_ERR_INVALID_ARG, "ldo=%lld < k*k", (long long)ldo);
  std::vector<std::pair<int64_t, int>> cols;
  for (int j = 0; j < n_mods; ++j) {
    const attr_module& m = mods[j];
    if (!m.a || !m.g || !m.R || !m.S) return fail(ATTR_ERR_INVALID_ARG, "module %d: NULL pointer", j);
    if (m.d_in <= 0 || m.d_out <= 0 || m.d_in > 65536 || m.d_out > 65536)
      return fail(ATTR_ERR_INVALID_ARG, "module %d: d_in=%lld d_out=%lld must be in [1, 65536]", j,
                  (long long)m.d_in, (long long)m.d_out);
    if (m.d_in % KS || m.d_out % KS)
      return fail(ATTR_ERR_ALIGNMENT, "module %d: d_in=%lld d_out=%lld must be multiples of %d", j,
                  (long long)m.d_in, (long long)m.d_out, KS);
    if (m.lda < m.d_in || m.ldg < m.d_out)
      return fail(ATTR_ERR_INVALID_ARG, "module %d: lda/ldg smaller than the row width", j);
    if (m.lda % ld_mult || m.ldg % ld_mult)
      return fail(ATTR_ERR_ALIGNMENT, "module %d: lda/ldg must be multiples of %d elements", j, ld_mult);
    if (!aligned16(m.a) || !aligned16(m.g) || !aligned16(m.R) || !aligned16(m.S))
      return fail(ATTR_ERR_ALIGNMENT, "module %d: pointers must be 16-byte aligned", j);
    if ((m.v_out == nullptr) != (m.v_in == nullptr))
      return fail(ATTR_ERR_INVALID_ARG, "module %d: v_out and v_in must both be set or both NULL", j);
    if ((reinterpret_cast<uintptr_t>(m.v_out) | reinterpret_cast<uintptr_t>(m.v_in)) & 3u)
      return fail(ATTR_ERR_ALIGNMENT, "module %d: v_out / v_in must be 4-byte aligned", j);
    if (m.lda * 256 * eb >= (1ll << 31) || m.ldg * 256 * eb >= (1ll << 31))
      return fail(ATTR_ERR_UNSUPPORTED, "module %d: row stride too large", j);
    if (m.out_col < 0 || m.out_col + kk > ldo)
      return fail(ATTR_ERR_INVALID_ARG, "module %d: out_col=%lld + k*k exceeds ldo=%lld", j,
                  (long long)m.out_col, (long long)ldo);
    cols.push_back({m.out_col, j});
  }
  std::sort(cols.begin(), cols.end());
  for (size_t j = 1; j < cols.size(); ++j)
    if (cols[j].first < cols[j - 1].first + kk)
      return fail(ATTR_ERR_INVALID_ARG, "modules %d and %d write overlapping output columns",
                  cols[j - 1].second, cols[j].second);
  return ATTR_OK;
}

}  // namespace

extern "C" {

const char* attr_last_error(void) { return g_err.c_str(); }

const char* attr_status_string(attr_status st) {
  switch (st) {
    case ATTR_OK: return "ATTR_OK";
    case ATTR_ERR_INVALID_ARG: return "ATTR_ERR_INVALID_ARG";
    case ATTR_ERR_UNSUPPORTED: return "ATTR_ERR_UNSUPPORTED";
    case ATTR_ERR_ALIGNMENT: return "ATTR_ERR_ALIGNMENT";
    case ATTR_ERR_WORKSPACE: return "ATTR_ERR_WORKSPACE";
    case ATTR_ERR_DEVICE: return "ATTR_ERR_DEVICE";
  }
  return "ATTR_UNKNOWN_STATUS";
}

int attr_abi_version(void) { return ATTR_ABI_VERSION; }

// ---------------------------------------------------------------------------
size_t attr_project_workspace_size(const attr_module* mods, int32_t n_mods, attr_dtype in_dtype,
                                   int64_t n_examples, int64_t T, int32_t k) {
  try {
    if (!mods || n_mods < 1 || n_mods > 4096 || (k != 16 && k != 32 && k != 64) || T < 1 ||
        n_examples < 0 || (in_dtype != ATTR_BF16 && in_dtype != ATTR_F32))
      return 0;
    return project_layout(mods, n_mods, dtype_bytes(in_dtype), n_examples, T, k).total;
  } catch (...) {
    return 0;
  }
}

// tok: per-token blocks into out rows [0, n_rows) (attr_project_tokens),
// else per-example rows (attr_project).
static attr_status project_impl(const attr_module* mods, int32_t n_mods, attr_dtype in_dtype,
                                int32_t k, int64_t n_examples, int64_t T,
                                const int64_t* row_offset, const int32_t* length, float* out,
                                int64_t ldo, void* ws, size_t ws_bytes, void* stream, bool tok,
                                int64_t n_rows) {
  try {
    g_err.clear();
    attr_status st = project_validate(mods, n_mods, in_dtype, k, n_examples, T, out, ldo);
    if (st != ATTR_OK) return st;
    if (tok && n_rows < 0) return fail(ATTR_ERR_INVALID_ARG, "n_rows=%lld is negative", (long long)n_rows);
    if (n_examples == 0) return ATTR_OK;
    const int eb = dtype_bytes(in_dtype);
    ProjLayout L = project_layout(mods, n_mods, eb, n_examples, T, k, tok);
    if (!ws || ws_bytes < L.total)
      return fail(ATTR_ERR_WORKSPACE, "attr_project needs %zu workspace bytes, got %zu", L.total,
                  ws ? ws_bytes : (size_t)0);
    if (reinterpret_cast<uintptr_t>(ws) & 255u)
      return fail(ATTR_ERR_ALIGNMENT, "workspace must be 256-byte aligned");
    const int64_t nblk = (int64_t)n_mods * L.n_chunks * n_examples;
    if (nblk > (1ll << 24))
      return fail(ATTR_ERR_UNSUPPORTED, "attr_project: %lld work items exceed one launch; split the batch",
                  (long long)nblk);
    hipStream_t s = static_cast<hipStream_t>(stream);
    char* base = static_cast<char*>(ws);
    attr::ProjTab* tab = reinterpret_cast<attr::ProjTab*>(base + L.off_tab);
    attr::ProjGroup* gtab = reinterpret_cast<attr::ProjGroup*>(base + L.off_gtab);
    char* pk = base + L.off_pk;
    float* part = reinterpret_cast<float*>(base + L.off_part);
    const bool bf16 = in_dtype == ATTR_BF16;
    const int nk = k / 16;
    for (int s0 = 0; s0 < n_mods; s0 += attr::kPackMax) {
      attr::PackArgs pa;
      std::memset(&pa, 0, sizeof(pa));
      pa.n = std::min(attr::kPackMax, n_mods - s0);
      pa.slot0 = s0;
      for (int j = 0; j < pa.n; ++j) {
        const attr_module& m = mods[L.order[s0 + j]];
        attr::PackEntry& e = pa.e[j];
        e.a = m.a;
        e.g = m.g;
        e.R = m.R;
        e.S = m.S;
        e.lda = m.lda;
        e.ldg = m.ldg;
        e.out_col = m.out_col;
        e.pk_off = (int64_t)L.pk_off[s0 + j];
        e.d_in = (int32_t)m.d_in;
        e.d_out = (int32_t)m.d_out;
        e.v_out = m.v_out;
        e.v_in = m.v_in;
        e.grp = L.slot_grp[s0 + j];
        e.lead_ms = L.lead_ms[s0 + j];
      }
      hipError_t e = attr::launch_project_pack(bf16, nk, pa, tab, gtab, pk, s);
      if (e != hipSuccess) return device_fail(e, "attr_project pack launch");
    }
    int32_t* wl_perm = nullptr;
    int32_t* wl_off = nullptr;
    if (attr::project_uses_worklist(length, n_examples, L.n_chunks)) {
      wl_perm = reinterpret_cast<int32_t*>(base + L.off_wl);
      wl_off = reinterpret_cast<int32_t*>(base + L.off_wl + align_up(4 * (size_t)n_examples));
    }
    hipError_t e = attr::launch_project_main(bf16, nk, tab, gtab, L.n_groups, L.n_chunks,
                                             n_examples, T, row_offset, length, wl_perm, wl_off,
                                             tok ? out : part, s, tok, ldo, n_rows);
    if (e != hipSuccess) return device_fail(e, "attr_project main launch");
    if (tok) return ATTR_OK;
    e = attr::launch_project_reduce(nk, tab, n_mods, L.n_chunks, n_examples, T, length, part, out,
                                    ldo, s);
    if (e != hipSuccess) return device_fail(e, "attr_project reduce launch");
    return ATTR_OK;
  } catch (const std::exception& ex) {
    return fail(ATTR_ERR_INVALID_ARG, "attr_project: host exception: %s", ex.what());
  } catch (...) {
    return fail(ATTR_ERR_INVALID_ARG, "attr_project: unknown host exception");
  }
}

attr_status attr_project(const attr_module* mods, int32_t n_mods, attr_dtype in_dtype, int32_t k,
                         int64_t n_examples, int64_t T, const int64_t* row_offset,
                         const int32_t* length, float* out, int64_t ldo, void* ws,
                         size_t ws_bytes, void* stream) {
  return project_impl(mods, n_mods, in_dtype, k, n_examples, T, row_offset, length, out, ldo, ws,
                      ws_bytes, stream, false, 0);
}

attr_status attr_project_tokens(const attr_module* mods, int32_t n_mods, attr_dtype in_dtype,
                                int32_t k, int64_t n_examples, int64_t T,
                                const int64_t* row_offset, const int32_t* length, float* out,
                                int64_t ldo, int64_t n_rows, void* ws, size_t ws_bytes,
                                void* stream) {
  return project_impl(mods, n_mods, in_dtype, k, n_examples, T, row_offset, length, out, ldo, ws,
                      ws_bytes, stream, true, n_rows);
}

attr_status attr_project_noalloc(const attr_module* mods, int32_t n_mods, attr_dtype in_dtype,
                                 int32_t k, int64_t n_examples, int64_t T,
                                 const int64_t* row_offset, const int32_t* length, float* out,
                                 int64_t ldo, void* stream) {
  try {
    g_err.clear();
    attr_status st = project_validate(mods, n_mods, in_dtype, k, n_examples, T, out, ldo);
    if (st != ATTR_OK) return st;
    if (n_examples == 0) return ATTR_OK;
    // the size check comes first: a call that cannot fit touches no device state
    const size_t need = project_layout(mods, n_mods, dtype_bytes(in_dtype), n_examples, T, k).total;
    if (need > attr::kProjectScratchBytes)
      return fail(ATTR_ERR_WORKSPACE,
                  "attr_project_noalloc: the call needs %zu bytes of scratch, the static buffer "
                  "holds %zu; split the batch or call attr_project with a workspace",
                  need, attr::kProjectScratchBytes);
    void* scratch = nullptr;
    const hipError_t e = attr::project_scratch(&scratch);
    if (e != hipSuccess) return device_fail(e, "attr_project_noalloc: static scratch address");
    return project_impl(mods, n_mods, in_dtype, k, n_examples, T, row_offset, length, out, ldo,
                        scratch, attr::kProjectScratchBytes, stream, false, 0);
  } catch (...) {
    return fail(ATTR_ERR_INVALID_ARG, "attr_project_noalloc: host exception");
  }
}

// ---------------------------------------------------------------------------
size_t attr_precond_accumulate_workspace_size(int64_t n_rows, int64_t D, attr_dtype x_dtype,
                                              attr_precond mode) {
  (void)x_dtype;
  if (n_rows <= 0 || D < 1) return 0;
  if (mode == ATTR_PRECOND_DIAG)
    return align_up((size_t)attr::colsumsq_panels(n_rows, D) * (size_t)D * sizeof(double));
  if (mode == ATTR_PRECOND_FULL) {
    const attr::SyrkPlan P = attr::plan_syrk(n_rows, D, 0);  // any stride's plan fits in it
    return align_up(P.part_bytes) + align_up(P.h64_bytes);
  }
  return 0;
}

attr_status attr_precond_accumulate(const void* X, attr_dtype x_dtype, int64_t n_rows, int64_t D,
                                    int64_t ldx, attr_precond mode, float* H, void* ws,
                                    size_t ws_bytes, void* stream) {
  try {
    g_err.clear();
    if (mode != ATTR_PRECOND_DIAG && mode != ATTR_PRECOND_FULL)
      return fail(ATTR_ERR_UNSUPPORTED, "attr_precond_accumulate: mode must be DIAG or FULL");
    if (!valid_dtype(x_dtype)) return fail(ATTR_ERR_UNSUPPORTED, "unknown x_dtype");
    const bool full = mode == ATTR_PRECOND_FULL;
    if (full && x_dtype == ATTR_F32)
      return fail(ATTR_ERR_UNSUPPORTED, "attr_precond_accumulate: FULL takes ATTR_F16 or ATTR_BF16 rows");
    if (n_rows < 0) return fail(ATTR_ERR_INVALID_ARG, "n_rows is negative");
    if (D < 1) return fail(ATTR_ERR_INVALID_ARG, "D must be >= 1");
    if (D % 8) return fail(ATTR_ERR_ALIGNMENT, "D=%lld must be a multiple of 8", (long long)D);
    if (ldx < D) return fail(ATTR_ERR_INVALID_ARG, "ldx < D");
    const int eb = dtype_bytes(x_dtype);
    if (ldx % (16 / eb)) return fail(ATTR_ERR_ALIGNMENT, "ldx must keep rows 16-byte aligned");
    if (!H) return fail(ATTR_ERR_INVALID_ARG, "H is NULL");
    if (n_rows > 0 && !X) return fail(ATTR_ERR_INVALID_ARG, "X is NULL");
    if (!aligned16(X) || !aligned16(H)) return fail(ATTR_ERR_ALIGNMENT, "X and H must be 16-byte aligned");
    if (full && D % 64) return fail(ATTR_ERR_ALIGNMENT, "FULL needs D a multiple of 64");
    if (full && D > 32768) return fail(ATTR_ERR_UNSUPPORTED, "FULL needs D <= 32768");
    if (full && ldx > 65536)
      return fail(ATTR_ERR_UNSUPPORTED, "FULL needs ldx <= 65536 (64-row stages of K-slices of at "
                  "least 16384 rows, each slice spanning at most 2 GiB)");
    if (overlap(span_of(X, n_rows, D, ldx, eb), span_of(H, full ? D : 1, D, D, 4)))
      return fail(ATTR_ERR_INVALID_ARG, "X and H overlap");
    if (n_rows == 0) return ATTR_OK;
    const size_t need = attr_precond_accumulate_workspace_size(n_rows, D, x_dtype, mode);
    if (!ws || ws_bytes < need)
      return fail(ATTR_ERR_WORKSPACE, "attr_precond_accumulate needs %zu workspace bytes", need);
    if (reinterpret_cast<uintptr_t>(ws) & 255u)
      return fail(ATTR_ERR_ALIGNMENT, "workspace must be 256-byte aligned");
    if (n_rows > (1ll << 40)) return fail(ATTR_ERR_UNSUPPORTED, "n_rows too large");
    hipError_t e;
    if (full) {
      const attr::SyrkPlan P = attr::plan_syrk(n_rows, D, ldx);
      if (P.Cs * ldx * 2 > (1ll << 31))
        return fail(ATTR_ERR_UNSUPPORTED, "internal: SYRK slice of %lld rows spans more than 2 GiB",
                    (long long)P.Cs);
      char* part = static_cast<char*>(ws);
      char* h64 = part + align_up(P.part_bytes);
      e = attr::launch_syrk(x_dtype == ATTR_BF16, X, ldx, n_rows, D, H, P, part, h64,
                            static_cast<hipStream_t>(stream));
    } else {
      e = attr::launch_colsumsq((int)x_dtype, X, ldx, n_rows, D, H, static_cast<double*>(ws),
                                static_cast<hipStream_t>(stream));
    }
    if (e != hipSuccess) return device_fail(e, "attr_precond_accumulate launch");
    return ATTR_OK;
  } catch (...) {
    return fail(ATTR_ERR_INVALID_ARG, "attr_precond_accumulate: host exception");
  }
}

// ---------------------------------------------------------------------------
size_t attr_precond_apply_workspace_size(int64_t n_rows, int64_t D, attr_precond mode) {
  if (mode != ATTR_PRECOND_FULL || n_rows <= 0 || D < 1) return 0;
  return attr::apply_full_workspace(n_rows, D, 1);
}

attr_status attr_precond_apply(const void* X, attr_dtype x_dtype, int64_t n_rows, int64_t D,
                               int64_t ldx, attr_precond mode, const float* M,
                               int32_t unit_normalize, void* Y, attr_dtype y_dtype, int64_t ldy,
                               void* ws, size_t ws_bytes, void* stream) {
  try {
    g_err.clear();
    if (mode != ATTR_PRECOND_NONE && mode != ATTR_PRECOND_DIAG && mode != ATTR_PRECOND_FULL)
      return fail(ATTR_ERR_UNSUPPORTED, "unknown preconditioner mode");
    if ((x_dtype != ATTR_F32 && x_dtype != ATTR_F16) || (y_dtype != ATTR_F32 && y_dtype != ATTR_F16))
      return fail(ATTR_ERR_UNSUPPORTED, "attr_precond_apply: dtypes must be ATTR_F32 or ATTR_F16");
    const bool full = mode == ATTR_PRECOND_FULL;
    if (full && x_dtype != ATTR_F16)
      return fail(ATTR_ERR_UNSUPPORTED, "attr_precond_apply: FULL takes ATTR_F16 rows");
    if (n_rows < 0) return fail(ATTR_ERR_INVALID_ARG, "n_rows is negative");
    if (D < 1) return fail(ATTR_ERR_INVALID_ARG, "D must be >= 1");
    if (D % 8) return fail(ATTR_ERR_ALIGNMENT, "D=%lld must be a multiple of 8", (long long)D);
    if (ldx < D || ldy < D) return fail(ATTR_ERR_INVALID_ARG, "ldx/ldy < D");
    const int xb = dtype_bytes(x_dtype), yb = dtype_bytes(y_dtype);
    if (ldx % (16 / xb) || ldy % (16 / yb))
      return fail(ATTR_ERR_ALIGNMENT, "ldx/ldy must keep rows 16-byte aligned");
    if (n_rows > 0 && (!X || !Y)) return fail(ATTR_ERR_INVALID_ARG, "X or Y is NULL");
    if (mode == ATTR_PRECOND_DIAG && !M) return fail(ATTR_ERR_INVALID_ARG, "DIAG needs M");
    if (full && !M) return fail(ATTR_ERR_INVALID_ARG, "FULL needs M");
    if (full && D % 64) return fail(ATTR_ERR_ALIGNMENT, "FULL needs D a multiple of 64");
    if (mode == ATTR_PRECOND_NONE && M) return fail(ATTR_ERR_INVALID_ARG, "NONE takes M = NULL");
    if (!aligned16(X) || !aligned16(Y) || !aligned16(M))
      return fail(ATTR_ERR_ALIGNMENT, "X, Y and M must be 16-byte aligned");
    const Span sx = span_of(X, n_rows, D, ldx, xb), sy = span_of(Y, n_rows, D, ldy, yb);
    const bool inplace = X == Y && x_dtype == y_dtype && ldx == ldy;
    if (!inplace && overlap(sx, sy)) return fail(ATTR_ERR_INVALID_ARG, "X and Y overlap");
    if (full && overlap(sx, sy)) return fail(ATTR_ERR_INVALID_ARG, "FULL cannot run in place");
    if (M && overlap(span_of(M, full ? D : 1, D, D, 4), sy))
      return fail(ATTR_ERR_INVALID_ARG, "M and Y overlap");
    if (n_rows == 0) return ATTR_OK;
    if (n_rows > (1ll << 31) - 1) return fail(ATTR_ERR_UNSUPPORTED, "n_rows exceeds one launch");
    if (full) {
      if (ldx * 256 * 2 >= (1ll << 31)) return fail(ATTR_ERR_UNSUPPORTED, "row stride too large");
      const size_t need = attr::apply_full_workspace(n_rows, D, unit_normalize ? 1 : 0);
      if (!ws || ws_bytes < need)
        return fail(ATTR_ERR_WORKSPACE, "attr_precond_apply (FULL) needs %zu workspace bytes", need);
      if (reinterpret_cast<uintptr_t>(ws) & 255u)
        return fail(ATTR_ERR_ALIGNMENT, "workspace must be 256-byte aligned");
      hipError_t e = attr::launch_apply_full(X, n_rows, ldx, D, M, (int)y_dtype, Y, ldy,
                                             unit_normalize ? 1 : 0, ws, static_cast<hipStream_t>(stream));
      if (e != hipSuccess) return device_fail(e, "attr_precond_apply (FULL) launch");
      return ATTR_OK;
    }
    hipError_t e = attr::launch_rowscale((int)x_dtype, (int)y_dtype, X, ldx, n_rows, D,
                                         mode == ATTR_PRECOND_DIAG ? M : nullptr, unit_normalize ? 1 : 0,
                                         nullptr, nullptr, 0, Y, ldy, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return device_fail(e, "attr_precond_apply launch");
    return ATTR_OK;
  } catch (...) {
    return fail(ATTR_ERR_INVALID_ARG, "attr_precond_apply: host exception");
  }
}

// ---------------------------------------------------------------------------
struct ScoreLayout {
  attr::ScorePlan plan;
  size_t off_s, off_i, off_p, total;
};

static ScoreLayout score_layout(int64_t n_q, int64_t n_g, int64_t D, int32_t k, int eb) {
  ScoreLayout L{};
  L.plan = attr::plan_score(n_q, n_g, D, k, eb);
  if (n_q <= 0 || n_g <= 0) return L;
  const size_t n = L.plan.list_entries;
  L.off_s = 0;
  L.off_i = align_up(n * sizeof(float));
  L.off_p = L.off_i + align_up(n * sizeof(int64_t));
  L.total = L.off_p + align_up(L.plan.spart_bytes);
  return L;
}

size_t attr_score_topk_workspace_size(int64_t n_q, int64_t n_g, int64_t D, int32_t k) {
  if (n_q < 0 || n_g < 0 || k < 1 || k > 128 || D < 1) return 0;
  // the fp16 plan needs at least as much workspace as the fp32 plan
  const ScoreLayout a = score_layout(n_q, n_g, D, k, 2), b = score_layout(n_q, n_g, D, k, 4);
  return a.total > b.total ? a.total : b.total;
}

attr_status attr_score_topk(const void* Q, int64_t n_q, int64_t ldq, const void* G, int64_t n_g,
                            int64_t ldg, attr_dtype dtype, int64_t D, int32_t k, int64_t index_base,
                            int32_t merge, float* top_score, int64_t* top_index, void* ws,
                            size_t ws_bytes, void* stream) {
  try {
    g_err.clear();
    if (dtype != ATTR_F16 && dtype != ATTR_F32)
      return fail(ATTR_ERR_UNSUPPORTED, "attr_score_topk: dtype must be ATTR_F16 or ATTR_F32");
    if (k < 1 || k > 128) return fail(ATTR_ERR_UNSUPPORTED, "attr_score_topk: k=%d must be in [1, 128]", k);
    if (n_q < 0 || n_g < 0) return fail(ATTR_ERR_INVALID_ARG, "n_q / n_g is negative");
    if (n_q > (1ll << 31) - 1 || n_g > (1ll << 31) - 1)
      return fail(ATTR_ERR_UNSUPPORTED, "n_q and n_g must be below 2^31 per call");
    if (D < 1) return fail(ATTR_ERR_INVALID_ARG, "D must be >= 1");
    const int eb = dtype_bytes(dtype);
    const int grp = dtype == ATTR_F16 ? 64 : 32;
    if (D % grp) return fail(ATTR_ERR_ALIGNMENT, "D=%lld must be a multiple of %d", (long long)D, grp);
    if (ldq < D || ldg < D) return fail(ATTR_ERR_INVALID_ARG, "ldq/ldg < D");
    if (ldq % (16 / eb) || ldg % (16 / eb))
      return fail(ATTR_ERR_ALIGNMENT, "ldq/ldg must keep rows 16-byte aligned");
    if (ldq * 256 * eb >= (1ll << 31) || ldg * 256 * eb >= (1ll << 31))
      return fail(ATTR_ERR_UNSUPPORTED, "row stride too large (256 rows must span < 2 GiB)");
    if (merge != 0 && merge != 1) return fail(ATTR_ERR_INVALID_ARG, "merge must be 0 or 1");
    if (index_base < 0 || index_base > (1ll << 62))
      return fail(ATTR_ERR_INVALID_ARG, "index_base must be in [0, 2^62]");
    if (n_q > 0 && (!Q || !top_score || !top_index))
      return fail(ATTR_ERR_INVALID_ARG, "Q / top_score / top_index is NULL");
    if (n_g > 0 && !G) return fail(ATTR_ERR_INVALID_ARG, "G is NULL");
    if (!aligned16(Q) || !aligned16(G) || !aligned16(top_score) || !aligned16(top_index))
      return fail(ATTR_ERR_ALIGNMENT, "Q, G, top_score and top_index must be 16-byte aligned");
    const Span ss = span_of(top_score, n_q, k, k, 4), si = span_of(top_index, n_q, k, k, 8);
    const Span sq = span_of(Q, n_q, D, ldq, eb), sg = span_of(G, n_g, D, ldg, eb);
    if (overlap(ss, si) || overlap(ss, sq) || overlap(ss, sg) || overlap(si, sq) || overlap(si, sg))
      return fail(ATTR_ERR_INVALID_ARG, "top_score / top_index overlap each other or the inputs");
    if (n_q == 0) return ATTR_OK;
    if (n_g == 0 && merge) return ATTR_OK;
    const ScoreLayout L = score_layout(n_q, n_g, D, k, eb);
    if (L.total > 0 && (!ws || ws_bytes < L.total))
      return fail(ATTR_ERR_WORKSPACE, "attr_score_topk needs %zu workspace bytes", L.total);
    if (reinterpret_cast<uintptr_t>(ws) & 255u)
      return fail(ATTR_ERR_ALIGNMENT, "workspace must be 256-byte aligned");
    char* base = static_cast<char*>(ws);
    hipError_t e = attr::launch_score_topk(
        dtype == ATTR_F16, L.plan, Q, n_q, ldq, G, n_g, ldg, k, index_base, merge, top_score,
        top_index, base ? reinterpret_cast<float*>(base + L.off_s) : nullptr,
        base ? reinterpret_cast<int64_t*>(base + L.off_i) : nullptr,
        base ? reinterpret_cast<float*>(base + L.off_p) : nullptr, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return device_fail(e, "attr_score_topk launch");
    return ATTR_OK;
  } catch (...) {
    return fail(ATTR_ERR_INVALID_ARG, "attr_score_topk: host exception");
  }
}

// ---------------------------------------------------------------------------
attr_status attr_probe_read(const void* x, size_t bytes, void* sink, void* stream) {
  g_err.clear();
  if (bytes == 0) return ATTR_OK;
  if (!x || !sink) return fail(ATTR_ERR_INVALID_ARG, "attr_probe_read: NULL pointer");
  if (!aligned16(x) || bytes % 16) return fail(ATTR_ERR_ALIGNMENT, "attr_probe_read: x and bytes must be 16-byte multiples");
  const hipError_t e = attr::launch_probe_read(x, bytes, sink, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ATTR_OK : device_fail(e, "attr_probe_read launch");
}

attr_status attr_probe_mfma(int64_t n_mfma, void* sink, void* stream) {
  g_err.clear();
  if (n_mfma <= 0 || n_mfma % 8) return fail(ATTR_ERR_INVALID_ARG, "attr_probe_mfma: n_mfma must be a positive multiple of 8");
  if (!sink) return fail(ATTR_ERR_INVALID_ARG, "attr_probe_mfma: NULL sink");
  const hipError_t e = attr::launch_probe_mfma(n_mfma, sink, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ATTR_OK : device_fail(e, "attr_probe_mfma launch");
}

}  // extern "C"
