// Declarations shared by the Sinkhorn translation units: constants, problem
// classes, the kernel parameters, the cross-lane helpers of the register
// paths and the launchers of the register kernels (one unit each).
#pragma once

#include "common.h"

namespace taot {

// Parameters of every Sinkhorn kernel of one call.
struct SkParams {
  const float* a;
  const float* b;
  int32_t B, R;
  const float* C;
  int64_t C_stride;
  float eps;
  int32_t iters;
  uint32_t flags;
  float* T;
  float* f;
  float* g;
  uint32_t* status;
  int32_t* stream_flag;  // [B] 1 = problem left to the streamed kernel
  float* kt_ws;          // streamed Kt storage, kt_stride floats per problem
  int64_t kt_stride;
  int32_t lds_kt_cap;    // Kt capacity (floats) of the LDS kernel
  int32_t all_streamed;  // every problem goes to the streamed kernel
  const int32_t* cbad;   // [matrices][cchunks] 1 = the chunk of C holds a non-finite entry
  int32_t cchunks;       // chunks of kScanChunk entries per cost matrix
  float* dn_ws;          // dense streamed iterate: per-problem state, dn_stride floats each
  int64_t dn_stride;
};

namespace {

constexpr int kSkThreads = 256;
constexpr int kSkWaves = kSkThreads / kWave;
constexpr int kSkStreamThreads = 1024;  // threads per problem of the streamed kernel
constexpr float kLo = 0x1p-60f;
constexpr float kHi = 0x1p60f;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kLdsMaxR = 256;            // beyond this every problem is streamed
constexpr int kVecArrays = 11;           // per-problem vectors of length R in LDS

__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float flog2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float frcp(float x) { return __builtin_amdgcn_rcpf(x); }

// Register classes: CPL columns per lane (|C| <= 64*CPL) and 8*C8 rows
// (|H| <= 8*C8).  Class 0 is every other problem (degenerate, larger, or the
// register path switched off).
__host__ __device__ constexpr int cpl_index(int cpl) { return cpl == 1 ? 0 : cpl == 2 ? 1 : 2; }
__host__ __device__ constexpr int wave_class(int cpl, int c8) { return 1 + cpl_index(cpl) * 8 + (c8 - 1); }
__device__ __forceinline__ int classify(int32_t nh, int32_t nc, uint32_t flags) {
  if (nh <= 0 || nc <= 0 || nh > 64 || nc > 256) return 0;
  if (flags & (TAOT_SK_FORCE_STREAM | TAOT_SK_NO_REGISTER)) return 0;
  const int cpl = nc <= 64 ? 1 : nc <= 128 ? 2 : 4;
  return wave_class(cpl, (nh + 7) / 8);
}

// Wide register classes (see the wide register path below): up to 96 hot
// and 1024 cold ranks, for problems no register class takes.
constexpr int kWideWaves = 12;
constexpr int kWideRows = 8 * kWideWaves;  // hot ranks
constexpr int kWideMaxCpl = 16;            // LDS slots per lane
constexpr int kWideCols = 64 * 15;         // cold ranks (15 columns per lane)
constexpr int kWideThreads = kWideWaves * kWave;
constexpr int kWideClassBase = 32;         // class codes 32 + CPL

// Columns per lane: 4, an even count up to 14, or 15.
__host__ __device__ constexpr int wide_cpl(int32_t nc) {
  return nc <= 256 ? 4 : nc > 896 ? 15 : (int)((nc + 127) / 128) * 2;
}
__device__ __forceinline__ int wide_class(int32_t nh, int32_t nc, uint32_t flags) {
  if (nh <= 0 || nc <= 0 || nh > kWideRows || nc > kWideCols) return 0;
  if (flags & (TAOT_SK_FORCE_STREAM | TAOT_SK_NO_REGISTER)) return 0;
  if (classify(nh, nc, flags) != 0) return 0;  // a register class takes it
  return kWideClassBase + wide_cpl(nc);
}
__host__ __device__ constexpr bool is_reg_class(int32_t c) { return c >= 1 && c < kWideClassBase; }
__host__ __device__ constexpr bool is_wide_class(int32_t c) { return c > kWideClassBase; }

// ---------------------------------------------------------------------------
// Register-resident path.  A problem's |H| x |C| block of Kt lives in the
// VGPRs of NW waves of one workgroup (NW = 1, 2 or 4).  Lane l of every wave
// owns compact columns l, l+64, ... (CPL of them); wave w holds the rows of
// chunks w*C8W .. w*C8W + C8W-1 (8 rows per chunk).
//   row half-step:    p_i = sum_c Kt_ic v_c per lane, then a transposed
//                     butterfly reduce-scatter over the 64 lanes (8 rows at a
//                     time: permlane32/16 swaps, then DPP) leaves the total of
//                     row 8q + (l >> 3) in lane l; rows never leave their wave.
//   column half-step: x_c = sum_i u_i Kt_ic over the wave's rows, the row
//                     scalings broadcast through LDS; with NW > 1 the waves'
//                     partial sums meet in LDS (one barrier per iteration) and
//                     are added in wave order, so every wave derives the same
//                     v and takes the same branches.
// An out-of-range scaling triggers the exact log-domain update of the wave's
// rows (or of all columns), absorbed into the potentials, with Kt rebuilt.
//
// Launch shape.  One kernel runs every register problem of a batch.  Its
// shapes use W waves per multi-wave problem (W = 4 when the batch is small
// enough that every problem can hold four waves at once, else W = 2), and its
// workgroups run either one problem on W waves ("multi") or one problem per
// wave ("single"), never two multi-wave problems, so workgroup barriers only
// ever join the waves of one problem.  Single groups of the two-wave shapes
// span a whole compute unit (eight waves) so that the problems sharing a SIMD
// can be paired by work.
//   W = 4 (at most 128 VGPRs, four waves per SIMD): problems of one chunk are
//     single; the rest are multi with ceil(C8 / 4) chunks per wave.
//   W = 2 (at most 256 VGPRs, two waves per SIMD): a problem is single when
//     its block fits one wave's 192 Kt registers, else (4 columns per lane and
//     more than 48 hot ranks) multi with ceil(C8 / 2) chunks per wave.
// Small batches thus spread a problem over more waves (a shorter dependent
// chain per wave, more waves per SIMD), while a batch that fills the chip
// with one wave per problem avoids the per-iteration exchange.

__host__ __device__ constexpr int max_c8_single(int W, int cpl) {
  return W == 4 ? 1 : (192 / (8 * cpl) < 8 ? 192 / (8 * cpl) : 8);
}
__host__ __device__ constexpr bool is_single(int W, int cpl, int c8) { return c8 <= max_c8_single(W, cpl); }
__host__ __device__ constexpr int c8_per_wave(int W, int cpl, int c8) {
  return is_single(W, cpl, c8) ? c8 : (c8 + W - 1) / W;
}
// Shapes compiled into the W-wave kernel for NW = 1 (single) or NW = W.
__host__ __device__ constexpr bool shape_ok(int W, int nw, int cpl, int c8w) {
  return nw == 1 ? c8w >= 1 && c8w <= max_c8_single(W, cpl)
                 : nw == W && (W == 4 ? c8w >= 1 && c8w <= 2 : cpl == 4 && c8w == 4);
}
__host__ __device__ constexpr bool shapes_covered() {
  for (int W = 2; W <= 4; W += 2)
    for (int ci = 0; ci < 3; ++ci)
      for (int c8 = 1; c8 <= 8; ++c8) {
        const int cpl = 1 << ci;
        const int nw = is_single(W, cpl, c8) ? 1 : W;
        if (!shape_ok(W, nw, cpl, c8_per_wave(W, cpl, c8))) return false;
      }
  return true;
}
static_assert(shapes_covered(), "every register class must map to a compiled shape");

// Decoded register class.
__device__ __forceinline__ int class_cpl(int32_t cls) { return 1 << ((cls - 1) / 8); }
__device__ __forceinline__ int class_c8(int32_t cls) { return (cls - 1) % 8 + 1; }

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  // every lane has a source lane for the patterns used here, so bound_ctrl
  // changes nothing but lets the move fold into the add
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, true));
}
__device__ __forceinline__ void swap32(float& lo, float& hi) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(lo), __float_as_uint(hi), false, false);
  lo = __uint_as_float(r[0]);
  hi = __uint_as_float(r[1]);
}
__device__ __forceinline__ void swap16(float& lo, float& hi) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(lo), __float_as_uint(hi), false, false);
  lo = __uint_as_float(r[0]);
  hi = __uint_as_float(r[1]);
}

// Sums 8 per-lane values over the wave; lane l ends with the total of value
// (l >> 3).  Halving steps pair lanes l ^ 32 (permlane32 swap), l ^ 16
// (permlane16 swap) and l <-> 15 - l (row_mirror); the last three steps add
// over l <-> l ^ 7 (row_half_mirror), l ^ 2 and l ^ 1 (quad_perm).
__device__ __forceinline__ float reduce8(float (&p)[8], int lane) {
#pragma unroll
  for (int k = 0; k < 4; ++k) { swap32(p[k], p[k + 4]); p[k] = p[k] + p[k + 4]; }
#pragma unroll
  for (int k = 0; k < 2; ++k) { swap16(p[k], p[k + 2]); p[k] = p[k] + p[k + 2]; }
  const bool b3 = lane & 8;
  const float keep = b3 ? p[1] : p[0];
  const float send = b3 ? p[0] : p[1];
  float y = keep + dpp<0x140>(send);  // row_mirror
  y = y + dpp<0x141>(y);              // row_half_mirror
  y = y + dpp<0x4E>(y);               // quad_perm [2,3,0,1]
  y = y + dpp<0xB1>(y);               // quad_perm [1,0,3,2]
  return y;
}

// Max and sum over the 64 lanes, every lane getting the result (bitwise the
// same: each step combines symmetric partners): DPP steps within each
// 16-lane row, then the permlane16 and permlane32 swaps across rows.
__device__ __forceinline__ float lanes_max(float x) {
  x = fmaxf(x, dpp<0xB1>(x));   // quad_perm [1,0,3,2]
  x = fmaxf(x, dpp<0x4E>(x));   // quad_perm [2,3,0,1]
  x = fmaxf(x, dpp<0x141>(x));  // row_half_mirror
  x = fmaxf(x, dpp<0x140>(x));  // row_mirror
  float y = x;
  swap16(x, y);
  x = fmaxf(x, y);
  y = x;
  swap32(x, y);
  return fmaxf(x, y);
}
__device__ __forceinline__ float lanes_sum(float x) {
  x = x + dpp<0xB1>(x);
  x = x + dpp<0x4E>(x);
  x = x + dpp<0x141>(x);
  x = x + dpp<0x140>(x);
  float y = x;
  swap16(x, y);
  x = x + y;
  y = x;
  swap32(x, y);
  return x + y;
}

// LDS of the register kernels, per workgroup: floats sA, F, u [64], the
// waves' column potentials [NW][4][64] and column demands [NW][64][4], for
// NW > 1 the column exchange [2 parities][NW][4][64]; then ints: a flag [4],
// cpos, hpos [R], cidx [256], hidx [64].
__host__ __device__ constexpr size_t wave_lds_floats(int nw) {
  return (size_t)3 * 64 + (size_t)2 * nw * 4 * 64 + (nw > 1 ? (size_t)2 * nw * 4 * 64 : 0);
}
__host__ __device__ constexpr size_t wave_lds_bytes(int32_t R, int nw) {
  return wave_lds_floats(nw) * 4 + (size_t)(4 + 2 * R + 256 + 64) * 4;
}

// Synchronisation among the waves of one problem: the workgroup barrier when
// the problem has the whole workgroup; for a one-wave problem (possibly beside
// other one-wave problems of the workgroup) an LDS fence of the wave.
template <int NW>
__device__ __forceinline__ void psync() {
  if constexpr (NW > 1) {
    __syncthreads();
  } else {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  }
}

// LDS of one wave of a single item, rounded to 16 bytes.
__host__ __device__ constexpr size_t single_lds_bytes(int32_t R) { return (wave_lds_bytes(R, 1) + 15) / 16 * 16; }

}  // namespace

// The register kernel for W waves per multi-wave problem and G waves per
// workgroup, on every listed problem (one translation unit each).
taot_status launch_reg_w4g4(const SkParams& p, const int32_t* multi, const int32_t* single, const int32_t* counts,
                            hipStream_t stream);
taot_status launch_reg_w2g8(const SkParams& p, const int32_t* multi, const int32_t* single, const int32_t* counts,
                            hipStream_t stream);
taot_status launch_reg_w2g2(const SkParams& p, const int32_t* multi, const int32_t* single, const int32_t* counts,
                            hipStream_t stream);
// The dense streamed iterate (TAOT_SK_DENSE) and its per-problem state in the
// streamed-plan storage of the workspace.
taot_status launch_dense(const SkParams& p, hipStream_t stream);
size_t dense_state_floats(int32_t R);

}  // namespace taot
