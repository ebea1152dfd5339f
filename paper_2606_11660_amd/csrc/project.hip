// Per-example double-sided random projection of linear-layer gradients
// (Figure 1 caption; Appendix B, paragraph "Gradients"):
//     P_i = sum_{t < len_i} (R^T g_t)(S^T a_t)^T,   k x k per module,
// computed from the token rows a_t, g_t without forming the d_out x d_in
// per-example gradient.
//
// Design (HBM-bound: every a/g element is read once and used for 2k flops):
//  * One workgroup (4 waves) owns one (module group, token chunk, example)
//    item of 64*TT tokens, a quarter of the chunk's valid tokens per wave.
//    One launch covers every item: module groups (modules that share their
//    input rows) by decreasing work per token, then chunk, then example, so
//    the dispatcher hands out the most expensive items first.
//  * Stage 1 runs on the matrix cores: A_tile (16 tokens x K) times the
//    packed S fragment gives 16 tokens x 16 projected columns.  Every lane
//    loads 16 contiguous bytes of one token row per step through a
//    range-checked buffer resource sized to the valid tokens, so padded or
//    missing tokens read as exact zeros (NaN padding never enters).
//  * Stage 2 contracts the two 16x16 fp32 tiles over tokens with fp32 MFMA:
//    the C layout of stage 1 (lane = column + 16 * (token / 4), register =
//    token % 4) is directly the A/B operand layout of the 16x16x4 fp32 MFMA
//    when register q is fed as step q, so no data moves between lanes.
//  * The four wave partials are summed in LDS in a fixed order and written
//    as one fp32 k x k partial per item; a second kernel sums the chunks of
//    each (module, example) in chunk order into the output row
//    (deterministic, no atomics).
#include <mutex>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace attr {
namespace {

// Scratch of the allocation-free projection entry point: one copy per GPU,
// held from the library's first use on that GPU until the process ends.  In
// host code `scratch` names a host-side stand-in, never the device memory:
// its device address comes from hipGetSymbolAddress, per device.
static __device__ __align__(256) char scratch[kProjectScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

template <bool BF16>
struct ElemT;
template <>
struct ElemT<true> {
  using tag = Bf16Tag;
  static constexpr int bytes = 2;
};
template <>
struct ElemT<false> {
  using tag = F32Tag;
  static constexpr int bytes = 4;
};

// Token tiles (16 tokens) per wave and load steps kept in flight, per
// fragment width NK (k = 16 NK).
#ifndef ATTR_PROJ_TT1
#define ATTR_PROJ_TT1 4
#endif
#ifndef ATTR_PROJ_PD
#define ATTR_PROJ_PD 3
#endif
template <int NK>
struct Tiles {
  static constexpr int TT = NK == 1 ? ATTR_PROJ_TT1 : (NK == 2 ? 2 : 1);
  static constexpr int PD = ATTR_PROJ_PD;
};

// bf16 bit pattern <-> float (bf16 is the upper half of an fp32 pattern);
// float -> bf16 rounds to nearest even, NaN stays NaN
__device__ inline float bf16_value(uint16_t h) { return __builtin_bit_cast(float, (uint32_t)h << 16); }
__device__ inline uint16_t bf16_rne(float x) {
  const uint32_t b = __builtin_bit_cast(uint32_t, x);
  if ((b & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((b >> 16) | 0x40u);
  return (uint16_t)((b + 0x7fffu + ((b >> 16) & 1u)) >> 16);
}

// ---------------------------------------------------------------------------
// pack: S [d_in, k] and R [d_out, k] (row-major) into MFMA B fragments.
// Fragment (step ks, column tile ct) is 64 lanes x 16 bytes; lane
// (j = lane % 16, grp = lane / 16) holds rows KS*ks + E*grp + e (e < E) of
// column 16*ct + j, where E = 16 / elem_bytes and KS = 4 E.
// ---------------------------------------------------------------------------
template <bool BF16, int NK>
__global__ __launch_bounds__(256) void project_pack_kernel(PackArgs args, ProjTab* tab,
                                                           ProjGroup* gtab, char* pk_base) {
  using E_t = ElemT<BF16>;
  constexpr int E = 16 / E_t::bytes;
  constexpr int KS = 4 * E;
  constexpr int K = 16 * NK;
  const int j = blockIdx.x;
  if (j >= args.n) return;
  const PackEntry pe = args.e[j];
  char* pk = pk_base + pe.pk_off;
  // blockIdx.y splits a module's fragments over gridDim.y workgroups
  const int f0 = (int)(blockIdx.y * blockDim.x + threadIdx.x);
  const int fstep = (int)(gridDim.y * blockDim.x);
  if (blockIdx.y == 0 && threadIdx.x == 0) {
    ProjTab t;
    t.a = pe.a;
    t.g = pe.g;
    t.pk = pk;
    t.lda = pe.lda;
    t.ldg = pe.ldg;
    t.out_col = pe.out_col;
    t.d_in = pe.d_in;
    t.d_out = pe.d_out;
    tab[args.slot0 + j] = t;
    if (pe.lead_ms > 0) gtab[pe.grp] = ProjGroup{args.slot0 + j, pe.lead_ms};
  }
  // Optimizer-state normalisation (factored second moment v = v_out v_in^T
  // / sum(v_out)): G / sqrt(v) = D_out G D_in with D_out = diag(sqrt(sum /
  // v_out)), D_in = diag(v_in^{-1/2}), so R^T (G / sqrt(v)) S = (D_out R)^T
  // G (D_in S): R's row i and S's row j are scaled here; a factor that is
  // not positive zeroes its row.  The sum runs in fp64 in a fixed order.
  const bool norm = pe.v_out != nullptr;
  double vsum = 0.0;
  if (norm) {
    __shared__ double red[256];
    double acc = 0.0;
    for (int i = threadIdx.x; i < pe.d_out; i += blockDim.x) {
      const float x = pe.v_out[i];
      acc += x > 0.f ? (double)x : 0.0;
    }
    red[threadIdx.x] = acc;
    for (int w = 128; w >= 1; w >>= 1) {
      __syncthreads();
      if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    }
    __syncthreads();
    vsum = red[0];
  }
  auto row_scale = [&](int side, int row) -> float {
    const float x = side == 0 ? pe.v_in[row] : pe.v_out[row];
    if (!(x > 0.f)) return 0.f;
    return (float)(side == 0 ? 1.0 / sqrt((double)x) : sqrt(vsum / (double)x));
  };
  for (int side = 0; side < 2; ++side) {
    const int d = side == 0 ? pe.d_in : pe.d_out;
    const char* src = (const char*)(side == 0 ? pe.S : pe.R);
    char* dst = pk + (side == 0 ? 0 : (size_t)pe.d_in * K * E_t::bytes);
    const int n_frag16 = (d / KS) * NK * kWave;  // 16-byte fragments
    for (int f = f0; f < n_frag16; f += fstep) {
      const int lane = f % kWave;
      const int ct = (f / kWave) % NK;
      const int ks = f / (kWave * NK);
      const int col = 16 * ct + (lane & 15);
      const int row0 = KS * ks + E * (lane >> 4);
      i32x4 v;
      if (E_t::bytes == 2) {
        uint16_t h[8];
#pragma unroll
        for (int e = 0; e < 8; ++e)
          h[e] = *(const uint16_t*)(src + ((size_t)(row0 + e) * K + col) * 2);
        if (norm) {
#pragma unroll
          for (int e = 0; e < 8; ++e) h[e] = bf16_rne(bf16_value(h[e]) * row_scale(side, row0 + e));
        }
        v.x = (int32_t)(h[0] | ((uint32_t)h[1] << 16));
        v.y = (int32_t)(h[2] | ((uint32_t)h[3] << 16));
        v.z = (int32_t)(h[4] | ((uint32_t)h[5] << 16));
        v.w = (int32_t)(h[6] | ((uint32_t)h[7] << 16));
      } else {
        int32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          w[e] = *(const int32_t*)(src + ((size_t)(row0 + e) * K + col) * 4);
        if (norm) {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            w[e] = __builtin_bit_cast(int32_t, __builtin_bit_cast(float, w[e]) * row_scale(side, row0 + e));
        }
        v.x = w[0];
        v.y = w[1];
        v.z = w[2];
        v.w = w[3];
      }
      *(i32x4*)(dst + (size_t)f * 16) = v;
    }
  }
}

// ---------------------------------------------------------------------------
// main projection kernel
// ---------------------------------------------------------------------------
// Accumulate one side: acc[tt][ct] += X_tile(tt) * B(ct) over d.
//
// The token rows are read in K-groups of 128 bytes per row (two MFMA steps).
// Global loads are line-coalesced: 8 consecutive lanes read one full 128-byte
// row segment, so one instruction covers 8 rows.  The MFMA operand layout
// wants 16 different rows per quarter-wave instead, so each group passes
// through a per-wave 2 KB LDS tile: written with an XOR swizzle (chunk ^
// row % 8) and read back as MFMA fragments, both conflict-free.  PD groups
// of loads are kept in flight in a register ring (the loop is unrolled by
// PD so ring slots are compile-time registers).
// MS > 1: the same token rows against the projections of MS modules that
// share them (one read of the rows, MS sets of MFMAs).
template <typename Tag, int E, int NK, int TT, int PD, int MS>
__device__ inline void project_side(__amdgpu_buffer_rsrc_t rsrc, int64_t ld, int d,
                                    const i32x4* const (&pk)[MS], int lane,
                                    i32x4* __restrict__ xp, f32x4 (&acc)[MS][TT][NK]) {
  constexpr int KS = 4 * E;   // K elements per MFMA step (one 16-byte fragment)
  constexpr int EB = 16 / E;  // element bytes
  constexpr int KG = 2 * KS;  // K elements per group = 128 bytes per row
  const int lrow = lane >> 3, lch = lane & 7;
  const uint32_t ld_base = (uint32_t)((int64_t)lrow * ld * EB + lch * 16);
  const uint32_t half_stride = (uint32_t)(8 * ld * EB);
  const uint32_t tile_stride = (uint32_t)(16 * ld * EB);
  const int wslot = lrow * 8 + (lch ^ lrow);
  const int ri = lane & 15, rgrp = lane >> 4;
  const int rslot0 = ri * 8 + (rgrp ^ (ri & 7));
  const int rslot1 = ri * 8 + ((4 + rgrp) ^ (ri & 7));
  const int n_g = d / KG;

  // Token-row loads run PD groups ahead (HBM latency); the projection
  // fragments (L2 resident) run one group ahead.
  i32x4 abuf[PD][TT][2], bcur[MS][2][NK], bnxt[MS][2][NK];
  auto issue = [&](int grp, i32x4 (&ab)[TT][2]) {
    const uint32_t off = ld_base + (uint32_t)grp * 128u;
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      ab[tt][0] = load16_stream(rsrc, off + tt * tile_stride);
      ab[tt][1] = load16_stream(rsrc, off + tt * tile_stride + half_stride);
    }
  };
  auto issue_b = [&](int grp, i32x4 (&bb)[MS][2][NK]) {
#pragma unroll
    for (int m = 0; m < MS; ++m)
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int ct = 0; ct < NK; ++ct) bb[m][s][ct] = pk[m][((2 * grp + s) * NK + ct) * kWave + lane];
  };
#pragma unroll
  for (int u = 0; u < PD - 1; ++u)
    if (u < n_g) issue(u, abuf[u]);
  issue_b(0, bcur);

  for (int g0 = 0; g0 < n_g; g0 += PD) {
#pragma unroll
    for (int u = 0; u < PD; ++u) {
      const int grp = g0 + u;
      if (grp + PD - 1 < n_g) issue(grp + PD - 1, abuf[(u + PD - 1) % PD]);
      if (grp < n_g) {
        if (grp + 1 < n_g) issue_b(grp + 1, bnxt);
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) {
          xp[tt * 128 + wslot] = abuf[u][tt][0];
          xp[tt * 128 + 64 + wslot] = abuf[u][tt][1];
        }
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) {
          const i32x4 f0 = xp[tt * 128 + rslot0];
          const i32x4 f1 = xp[tt * 128 + rslot1];
#pragma unroll
          for (int m = 0; m < MS; ++m)
#pragma unroll
            for (int ct = 0; ct < NK; ++ct) {
              acc[m][tt][ct] = mma16(Tag{}, f0, bcur[m][0][ct], acc[m][tt][ct]);
              acc[m][tt][ct] = mma16(Tag{}, f1, bcur[m][1][ct], acc[m][tt][ct]);
            }
        }
#pragma unroll
        for (int m = 0; m < MS; ++m)
#pragma unroll
          for (int s = 0; s < 2; ++s)
#pragma unroll
            for (int ct = 0; ct < NK; ++ct) bcur[m][s][ct] = bnxt[m][s][ct];
      }
    }
  }
}

// f(integral_constant<int, I>) for I = B .. E - 1, in order.
template <int B, int E>
struct StaticFor {
  template <typename F>
  __device__ static inline void run(F&& f) {
    if constexpr (B < E) {
      f(std::integral_constant<int, B>{});
      StaticFor<B + 1, E>::run(f);
    }
  }
};

// v of lane N of this lane's row of 16 (DPP row_newbcast:N).
template <int N>
__device__ inline float row_bcast(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x150 + N, 0xf, 0xf, false));
}

// One (group, token chunk, example) item, run by one workgroup.  A group
// is MS modules (consecutive slots from s0) that share their input rows a:
// the a tiles are read once and projected through each member's S; each
// member's own g rows follow, and each member's k x k partial goes to its
// slot's item.
// TOK: per-token blocks instead of the token sum: token t's (R^T g_t)(S^T
// a_t)^T is written to row (first row of the example) + t of `partial`
// (then the caller's output, row stride ldo, n_rows rows), at the module's
// out_col; no partials, no reduction.
template <bool BF16, int NK, int MS, bool TOK>
__device__ inline void project_item(const ProjTab* __restrict__ tab, int s0, uint32_t i, int c,
                                    int n_chunks, int64_t n_ex, int64_t T, int64_t len,
                                    const int64_t* __restrict__ row_offset,
                                    float* __restrict__ partial, int64_t ldo, int64_t n_rows,
                                    i32x4* __restrict__ xpose, float* __restrict__ red) {
  using E_t = ElemT<BF16>;
  using Tag = typename E_t::tag;
  constexpr int EB = E_t::bytes;
  constexpr int E = 16 / EB;
  constexpr int KS = 4 * E;
  constexpr int TT = Tiles<NK>::TT;
  constexpr int TPW = 16 * TT;  // tokens per wave
  constexpr int CT = 4 * TPW;   // tokens per workgroup
  constexpr int KK = 256 * NK * NK;
  const int64_t t0 = (int64_t)c * CT;

  // The wave index is uniform per wave; readfirstlane lets the compiler keep
  // everything derived from it (token range, buffer resources) in SGPRs.
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63;
  // The chunk's valid tokens are spread evenly over the four waves (TPW each
  // in a full chunk), so the last, partial chunk of an example keeps every
  // wave busy for a quarter of it instead of leaving trailing waves idle
  // while the workgroup holds its slot.
  const int64_t nv = len - t0 < CT ? len - t0 : CT;  // > 0
  const int64_t q = (nv + 3) / 4;                     // <= TPW
  const int64_t wt0 = t0 + (int64_t)wave * q;
  int64_t ntok = nv - (int64_t)wave * q;
  ntok = ntok < 0 ? 0 : (ntok > q ? q : ntok);
  const int64_t row0 = ntok > 0 ? (row_offset ? row_offset[i] : (int64_t)i * T) + wt0 : 0;
  i32x4* xp = xpose + wave * (TT * 128);

  f32x4 At[MS][TT][NK];
#pragma unroll
  for (int m = 0; m < MS; ++m)
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
      for (int ct = 0; ct < NK; ++ct) At[m][tt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (ntok > 0) {
    const ProjTab m0 = tab[s0];
    const char* a_ptr = (const char*)m0.a + row0 * m0.lda * EB;
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(a_ptr, (uint32_t)(ntok * m0.lda * EB));
    const i32x4* pkS[MS];
#pragma unroll
    for (int m = 0; m < MS; ++m) pkS[m] = (const i32x4*)tab[s0 + m].pk;
    project_side<Tag, E, NK, TT, Tiles<NK>::PD, MS>(ra, m0.lda, m0.d_in, pkS, lane, xp, At);
  }

#pragma unroll
  for (int m = 0; m < MS; ++m) {
    f32x4 P[NK][NK];
#pragma unroll
    for (int rt = 0; rt < NK; ++rt)
#pragma unroll
      for (int ct = 0; ct < NK; ++ct) P[rt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (ntok > 0) {
      const ProjTab md = tab[s0 + m];
      const char* g_ptr = (const char*)md.g + row0 * md.ldg * EB;
      const __amdgpu_buffer_rsrc_t rg = make_rsrc(g_ptr, (uint32_t)(ntok * md.ldg * EB));
      const i32x4* pkR[1] = {(const i32x4*)md.pk + (size_t)(md.d_in / KS) * NK * kWave};
      f32x4 Gt[1][TT][NK];
#pragma unroll
      for (int tt = 0; tt < TT; ++tt)
#pragma unroll
        for (int ct = 0; ct < NK; ++ct) Gt[0][tt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
      project_side<Tag, E, NK, TT, Tiles<NK>::PD, 1>(rg, md.ldg, md.d_out, pkR, lane, xp, Gt);

      if constexpr (TOK) {
        // register q of the stage-1 tiles holds token 16 tt + 4 (lane / 16) +
        // q of the wave, column lane % 16: each 16-lane row writes its own
        // token's block, taking g~[t][r] from lane r % 16 of the row by a DPP
        // row broadcast (a VALU move: a shuffle through the LDS crossbar put
        // its latency between every product and its store)
#pragma unroll
        for (int tt = 0; tt < TT; ++tt)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int tw = 16 * tt + 4 * (lane >> 4) + q;
            if (tw < ntok && row0 + tw < n_rows) {  // whole 16-lane rows
              float* orow = partial + (row0 + tw) * ldo + md.out_col + (lane & 15);
              StaticFor<0, 16 * NK>::run([&](auto rc) {
                constexpr int r = decltype(rc)::value;
                const float gr = row_bcast<(r & 15)>(Gt[0][tt][r >> 4][q]);
#pragma unroll
                for (int ct = 0; ct < NK; ++ct)
                  __builtin_nontemporal_store(gr * At[m][tt][ct][q], orow + r * 16 * NK + 16 * ct);
              });
            }
          }
      } else {
        // P[r][c] += sum_tokens Gt[token][r] * At[token][c]; register q of the
        // stage-1 tiles holds token 4 * (lane / 16) + q, column lane % 16.
#pragma unroll
        for (int tt = 0; tt < TT; ++tt)
#pragma unroll
          for (int rt = 0; rt < NK; ++rt)
#pragma unroll
            for (int ct = 0; ct < NK; ++ct)
#pragma unroll
              for (int q = 0; q < 4; ++q)
                P[rt][ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(Gt[0][tt][rt][q], At[m][tt][ct][q],
                                                                 P[rt][ct], 0, 0, 0);
      }
    }
    if constexpr (TOK) continue;

    // Fixed-order reduction of the four wave partials: waves 1..3 park their
    // tiles in LDS, wave 0 adds them in wave order and writes the item.
    if (m > 0) __syncthreads();  // wave 0 has read the previous member's tiles
    if (wave > 0) {
#pragma unroll
      for (int rt = 0; rt < NK; ++rt)
#pragma unroll
        for (int ct = 0; ct < NK; ++ct)
#pragma unroll
          for (int q = 0; q < 4; ++q) red[(wave - 1) * KK + ((rt * NK + ct) * 4 + q) * kWave + lane] = P[rt][ct][q];
    }
    __syncthreads();
    if (wave == 0) {
      float* dst = partial + (((int64_t)(s0 + m) * n_chunks + c) * (int64_t)n_ex + i) * KK;
#pragma unroll
      for (int rt = 0; rt < NK; ++rt)
#pragma unroll
        for (int ct = 0; ct < NK; ++ct)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int e = ((rt * NK + ct) * 4 + q) * kWave + lane;
            float v = P[rt][ct][q];
            v += red[e];
            v += red[KK + e];
            v += red[2 * KK + e];
            dst[e] = v;
          }
    }
  }
}


// Work list of a call with per-example lengths (one workgroup): example i
// has n_i = ceil(len_i / CT) chunks.  perm lists the examples by decreasing
// n_i (the order within equal n_i is whatever the scatter gives: it only
// decides which workgroup takes an item, never a result), so the examples
// that have a chunk c are exactly perm[0 .. cnt_c), cnt_c = #{i : n_i > c};
// off[c] = cnt_0 + ... + cnt_{c-1} is the first item of chunk row c within a
// group and off[n_chunks] the items per group.
__global__ __launch_bounds__(1024) void project_worklist_kernel(const int32_t* __restrict__ length,
                                                                int64_t n_ex, int64_t T, int CT,
                                                                int n_chunks,
                                                                int32_t* __restrict__ perm,
                                                                int32_t* __restrict__ off) {
  __shared__ int hist[kWorklistMaxChunks + 1];
  __shared__ int cur[kWorklistMaxChunks + 1];
  for (int j = threadIdx.x; j <= n_chunks; j += 1024) hist[j] = 0;
  __syncthreads();
  auto chunks_of = [&](int64_t i) {
    int64_t len = length[i];
    len = len < 0 ? 0 : (len > T ? T : len);
    return (int)((len + CT - 1) / CT);
  };
  for (int64_t i = threadIdx.x; i < n_ex; i += 1024) atomicAdd(&hist[chunks_of(i)], 1);
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;  // examples with more chunks than n come first
    for (int n = n_chunks; n >= 0; --n) {
      cur[n] = run;
      run += hist[n];
    }
    int acc = 0;  // cnt_c = cur[c]: examples in buckets above c
    for (int c = 0; c < n_chunks; ++c) {
      off[c] = acc;
      acc += cur[c];
    }
    off[n_chunks] = acc;
  }
  __syncthreads();
  for (int64_t i = threadIdx.x; i < n_ex; i += 1024) perm[atomicAdd(&cur[chunks_of(i)], 1)] = (int32_t)i;
}

// One workgroup per (group, token chunk, example) item of the whole call:
// items are enumerated group major (groups in table order, largest work
// first), then chunk, then example, so the dispatcher hands out the most
// expensive items first and the cheapest fill the tail of the one launch.
// The group size is read from the group table and dispatched at run time
// (uniform per workgroup); every size fits two waves per SIMD.
template <bool BF16, int NK, bool TOK>
__global__ __launch_bounds__(256, 2) void project_main_kernel(
    const ProjTab* __restrict__ tab, const ProjGroup* __restrict__ gtab, int n_groups,
    int n_chunks, int64_t n_ex, int64_t T, const int64_t* __restrict__ row_offset,
    const int32_t* __restrict__ length, const int32_t* __restrict__ wl_perm,
    const int32_t* __restrict__ wl_off, float* __restrict__ partial, int64_t ldo,
    int64_t n_rows) {
  constexpr int TT = Tiles<NK>::TT;
  constexpr int CT = 4 * 16 * TT;  // tokens per workgroup
  constexpr int KK = 256 * NK * NK;
  // Work-item decode in 32-bit scalar arithmetic (the host keeps the grid
  // below 2^24 items and n_examples below 2^31).  Workgroups go to the 8
  // XCDs round robin (block % 8), so the decode must not tie an example to
  // an XCD: with the example index varying fastest, example i would run on
  // XCD i % 8 for the whole call and each XCD would carry the summed length
  // of its own examples (ragged batches left XCDs idle while others worked).
  const uint32_t blk = blockIdx.x;
  uint32_t i;
  int c;
  ProjGroup gr;
  if (wl_perm) {
    // work list: block b takes the b-th valid item (group major, then chunk
    // row, then examples longest first); the blocks past the last item exit
    const uint32_t per = (uint32_t)wl_off[n_chunks];
    if (per == 0) return;
    const uint32_t g = blk / per;
    if (g >= (uint32_t)n_groups) return;  // uniform over the workgroup
    const uint32_t r = blk - g * per;
    int lo = 0, hi = n_chunks - 1;  // largest c with off[c] <= r
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if ((uint32_t)wl_off[mid] <= r) lo = mid;
      else hi = mid - 1;
    }
    c = lo;
    i = (uint32_t)wl_perm[r - (uint32_t)wl_off[c]];
    gr = gtab[g];
  } else {
    // dense decode: the example index is rotated per (group, chunk) row so
    // that every XCD takes every example equally often
    const uint32_t nex = (uint32_t)n_ex;
    const uint32_t rest = blk / nex;
    const uint32_t rot = rest + rest / (uint32_t)n_chunks;
    i = (blk % nex + rot % nex) % nex;
    c = (int)(rest % (uint32_t)n_chunks);
    gr = gtab[rest / (uint32_t)n_chunks];
  }

  int64_t len = length ? (int64_t)length[i] : T;
  len = len < 0 ? 0 : (len > T ? T : len);
  if ((int64_t)c * CT >= len) return;  // uniform over the workgroup

  __shared__ i32x4 xpose[4 * TT * 128];
  __shared__ float red[3 * KK];
  // groups of three at k = 64 and grouped per-token blocks would pass 256
  // VGPRs; the host never forms them
  constexpr bool m2 = !TOK;
  constexpr bool m3 = !TOK && NK < 4;
  if (m3 && gr.ms == 3)
    project_item<BF16, NK, (m3 ? 3 : 1), TOK>(tab, gr.slot0, i, c, n_chunks, n_ex, T, len,
                                               row_offset, partial, ldo, n_rows, xpose, red);
  else if (m2 && gr.ms == 2)
    project_item<BF16, NK, (m2 ? 2 : 1), TOK>(tab, gr.slot0, i, c, n_chunks, n_ex, T, len,
                                               row_offset, partial, ldo, n_rows, xpose, red);
  else
    project_item<BF16, NK, 1, TOK>(tab, gr.slot0, i, c, n_chunks, n_ex, T, len, row_offset,
                                   partial, ldo, n_rows, xpose, red);
}

// ---------------------------------------------------------------------------
// reduce: out[i, out_col + r*k + c] = sum over chunks of the item partials.
// Partial element e = ((rt*NK + ct)*4 + q)*64 + lane holds
// r = 16 rt + 4 (lane / 16) + q, c = 16 ct + lane % 16.
// ---------------------------------------------------------------------------
template <int NK>
__global__ __launch_bounds__(256) void project_reduce_kernel(
    const ProjTab* __restrict__ tab, int n_chunks, int64_t n_ex, int64_t T, int CT,
    const int32_t* __restrict__ length, const float* __restrict__ partial,
    float* __restrict__ out, int64_t ldo) {
  constexpr int K = 16 * NK;
  constexpr int KK = K * K;
  const int64_t i = blockIdx.x % n_ex;
  const int s = (int)(blockIdx.x / n_ex);
  int64_t len = length ? (int64_t)length[i] : T;
  len = len < 0 ? 0 : (len > T ? T : len);
  const int nck = (int)((len + CT - 1) / CT);
  const int64_t out_col = tab[s].out_col;
  for (int e = threadIdx.x; e < KK; e += blockDim.x) {
    float v = 0.f;
    for (int c = 0; c < nck; ++c) v += partial[((((int64_t)s * n_chunks + c) * n_ex) + i) * KK + e];
    const int lane = e & 63;
    const int q = (e >> 6) & 3;
    const int tile = e >> 8;
    const int rt = tile / NK, ct = tile % NK;
    const int r = 16 * rt + 4 * (lane >> 4) + q;
    const int cc = 16 * ct + (lane & 15);
    out[i * ldo + out_col + r * K + cc] = v;
  }
}

}  // namespace

hipError_t project_scratch(void** ptr) {
  *ptr = nullptr;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));  // the current device's copy
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

int project_chunk_tokens(int nk) {
  return 64 * (nk == 1 ? ATTR_PROJ_TT1 : (nk == 2 ? 2 : 1));
}

size_t project_packed_bytes(int64_t d_in, int64_t d_out, int k, int elem_bytes) {
  return (size_t)(d_in + d_out) * (size_t)k * (size_t)elem_bytes;
}

hipError_t launch_project_pack(bool bf16, int nk, const PackArgs& args, ProjTab* tab,
                               ProjGroup* gtab, char* pk_base, hipStream_t s) {
  dim3 grid(args.n, 8), block(256);
#define ATTR_PACK(B, N) \
  hipLaunchKernelGGL((project_pack_kernel<B, N>), grid, block, 0, s, args, tab, gtab, pk_base)
  if (bf16) {
    if (nk == 1) ATTR_PACK(true, 1);
    else if (nk == 2) ATTR_PACK(true, 2);
    else ATTR_PACK(true, 4);
  } else {
    if (nk == 1) ATTR_PACK(false, 1);
    else if (nk == 2) ATTR_PACK(false, 2);
    else ATTR_PACK(false, 4);
  }
#undef ATTR_PACK
  return hipGetLastError();
}

hipError_t launch_project_main(bool bf16, int nk, const ProjTab* tab, const ProjGroup* gtab,
                               int n_groups, int n_chunks, int64_t n_ex, int64_t T,
                               const int64_t* row_offset, const int32_t* length,
                               int32_t* wl_perm, int32_t* wl_off,
                               float* partial, hipStream_t s, bool tok, int64_t ldo,
                               int64_t n_rows) {
  const int64_t nblk = (int64_t)n_groups * n_chunks * n_ex;
  if (nblk == 0) return hipSuccess;
  if (wl_perm) {
    hipLaunchKernelGGL(project_worklist_kernel, dim3(1), dim3(1024), 0, s, length, n_ex, T,
                       project_chunk_tokens(nk), n_chunks, wl_perm, wl_off);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  dim3 grid((unsigned)nblk), block(256);
#define ATTR_MAIN(B, N, TK)                                                                   \
  hipLaunchKernelGGL((project_main_kernel<B, N, TK>), grid, block, 0, s, tab, gtab, n_groups, \
                     n_chunks, n_ex, T, row_offset, length, (const int32_t*)wl_perm,          \
                     (const int32_t*)wl_off, partial, ldo, n_rows)
#define ATTR_MAIN_TK(B, N) \
  if (tok) ATTR_MAIN(B, N, true); \
  else ATTR_MAIN(B, N, false);
  if (bf16) {
    if (nk == 1) { ATTR_MAIN_TK(true, 1) }
    else if (nk == 2) { ATTR_MAIN_TK(true, 2) }
    else { ATTR_MAIN_TK(true, 4) }
  } else {
    if (nk == 1) { ATTR_MAIN_TK(false, 1) }
    else if (nk == 2) { ATTR_MAIN_TK(false, 2) }
    else { ATTR_MAIN_TK(false, 4) }
  }
#undef ATTR_MAIN_TK
#undef ATTR_MAIN
  return hipGetLastError();
}

hipError_t launch_project_reduce(int nk, const ProjTab* tab, int n_slots, int n_chunks,
                                 int64_t n_ex, int64_t T, const int32_t* length,
                                 const float* partial, float* out, int64_t ldo,
                                 hipStream_t s) {
  dim3 grid((unsigned)((int64_t)n_slots * n_ex)), block(256);
  const int CT = project_chunk_tokens(nk);
#define ATTR_RED(N)                                                                          \
  hipLaunchKernelGGL((project_reduce_kernel<N>), grid, block, 0, s, tab, n_chunks, n_ex, T, CT, \
                     length, partial, out, ldo)
  if (nk == 1) ATTR_RED(1);
  else if (nk == 2) ATTR_RED(2);
  else ATTR_RED(4);
#undef ATTR_RED
  return hipGetLastError();
}

}  // namespace attr
