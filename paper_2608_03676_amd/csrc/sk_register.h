// Register-resident Sinkhorn path: the per-wave solvers (full-wave and
// folded layouts), the per-problem dispatch and the register kernel,
// included by the translation unit of each kernel instance.
#pragma once

#include "sk_common.h"

namespace taot {
namespace {

// Iterations and outputs of one problem on NW waves of CPL columns per lane
// and C8W chunks per wave; the caller has filled the LDS vectors and the
// first-update potentials Fl.
template <int CPL, int C8W, int NW, int WV>
__device__ __forceinline__ void wave_solve(const SkParams& p, int64_t pb, int32_t nh, int32_t nc,
                                           const int32_t* cpos, const int32_t* hpos, const int32_t* cidx,
                                           const int32_t* hidx, const float* sAl, float* Fl, float* ul,
                                           float* Gall, float* Sall, float* xbuf, float kappa) {
  constexpr int MW = 8 * C8W;  // rows per wave
  const int lane = threadIdx.x & (kWave - 1);
  constexpr int wv = WV;  // this wave (a compile-time constant, so per-wave LDS offsets are immediates)
  constexpr int rb = MW * wv;  // first row of this wave
  const int32_t R = p.R;
  const float* bd = p.b + pb * R;
  const float* Cb = p.C + pb * p.C_stride;
  // the column potentials G (log2 units) are only touched by the log-domain
  // updates: they live in this wave's LDS slice, one value per lane and column
  float* Gw = Gall + wv * 4 * kWave + lane;
  // the column demands, read once per iteration: this wave's slice, the
  // lane's CPL values contiguous
  float* Sw = Sall + (wv * kWave + lane) * 4;
#define CV(c) (lane + kWave * (c) < nc)
#define CJ(c) (CV(c) ? cidx[lane + kWave * (c)] : 0)
#define RV(q) (rb + 8 * (q) + (lane >> 3) < nh)
#define GL(c) Gw[(c) * kWave]

  float K[MW][CPL];
  float v[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    Sw[c] = CV(c) ? bd[CJ(c)] : 0.f;
    v[c] = CV(c) ? 1.f : 0.f;
    GL(c) = 0.f;
  }
  // the lane's column demands (padding columns 0)
  auto demands = [&](float (&sB)[CPL]) {
    if constexpr (CPL == 4) {
      const float4 d = *reinterpret_cast<const float4*>(Sw);
      sB[0] = d.x; sB[1] = d.y; sB[2] = d.z; sB[3] = d.w;
    } else if constexpr (CPL == 2) {
      const float2 d = *reinterpret_cast<const float2*>(Sw);
      sB[0] = d.x; sB[1] = d.y;
    } else {
      sB[0] = Sw[0];
    }
  };
  // Kt of this wave's rows from the potentials (after the exact log-domain
  // update of each row's potential when row_update is set:
  // F_i = log2 s~_i - LSE2_c(G_c + log2 v_c - C'_ic), absorbing u_i).  Each
  // row's support index is read at an opaque position, so that the row's cost
  // address is formed here and not kept in registers for the whole iteration
  // loop.
  auto build = [&](bool row_update) {
#pragma unroll
    for (int i = 0; i < MW; ++i) {
      const int gi = rb + i;
      if (gi < nh) {
        int32_t go = __builtin_amdgcn_readfirstlane(gi);
        asm volatile("" : "+s"(go));
        const float* crow = Cb + (int64_t)__builtin_amdgcn_readfirstlane(hidx[go]) * R;
        float cc[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) cc[c] = CV(c) ? crow[CJ(c)] * kappa : 0.f;
        float fi;
        if (row_update) {
          float t[CPL];
          float mx = -INFINITY;
#pragma unroll
          for (int c = 0; c < CPL; ++c) {
            t[c] = CV(c) ? (GL(c) + flog2(v[c])) - cc[c] : -INFINITY;
            mx = fmaxf(mx, t[c]);
          }
          mx = lanes_max(mx);
          float sum = 0.f;
#pragma unroll
          for (int c = 0; c < CPL; ++c) sum += CV(c) ? fexp2(t[c] - mx) : 0.f;
          sum = lanes_sum(sum);
          fi = flog2(sAl[gi]) - (mx + flog2(sum));
          if (lane == 0) Fl[gi] = fi;
        } else {
          fi = Fl[gi];
        }
#pragma unroll
        for (int c = 0; c < CPL; ++c) K[i][c] = CV(c) ? fexp2((fi + GL(c)) - cc[c]) : 0.f;
      } else {
#pragma unroll
        for (int c = 0; c < CPL; ++c) K[i][c] = 0.f;
      }
    }
  };

  // The row scalings live in LDS (ul): lane l computes that of row
  // rb + 8q + (l >> 3) of chunk q, and lanes l = 8k store them.
#define UST(q, val) \
  if ((lane & 7) == 0) ul[rb + 8 * (q) + (lane >> 3)] = (val)
#pragma unroll
  for (int q = 0; q < C8W; ++q) UST(q, RV(q) ? 1.f : 0.f);
  // the scaled supply of the lane's row of each chunk, held in registers
  float sAq[C8W];
#pragma unroll
  for (int q = 0; q < C8W; ++q) sAq[q] = sAl[rb + 8 * q + (lane >> 3)];

  // The iterations run in an inner loop that only ever reads Kt.  An
  // out-of-range scaling leaves it; the log-domain update is then taken and Kt
  // rebuilt before the iterations resume, so Kt is never live across an update.
  int32_t it = 1;
  bool skip_row = true;     // iteration 1 has no row half-step (u follows from v = 1)
  bool row_update = false;  // this wave's rows take the log-domain update first
  for (;;) {
    build(row_update);
    if (row_update) {
#pragma unroll
      for (int q = 0; q < C8W; ++q) UST(q, RV(q) ? 1.f : 0.f);
      row_update = false;
    }
    bool done = false, col_fail = false;
    for (;;) {
      if (!skip_row) {
        // ---- row half-step on this wave's rows: u_i = s~_i / sum_c Kt_ic v_c ---------
        // padding rows (all-zero Kt) divide by 1 and count as 1 in the range test
        uint32_t lo = 0xFFFFFFFFu, hi = 0u;  // range of the scalings' bit patterns
#define TAOT_ROW_SUMS(q, pp)                                                                          \
  _Pragma("unroll") for (int r = 0; r < 8; ++r) {                                                     \
    float acc = K[8 * (q) + r][0] * v[0];                                                             \
    _Pragma("unroll") for (int c = 1; c < CPL; ++c) acc = __builtin_fmaf(K[8 * (q) + r][c], v[c], acc); \
    pp[r] = acc;                                                                                      \
  }
#define TAOT_ROW_FINISH(q, y)                                                                         \
  {                                                                                                   \
    const bool rv = RV(q);                                                                            \
    const float un = sAq[q] * frcp(rv ? (y) : 1.f);                                                   \
    const uint32_t bits = __float_as_uint(rv ? un : 1.f);                                             \
    lo = bits < lo ? bits : lo;                                                                       \
    hi = bits > hi ? bits : hi;                                                                       \
    UST(q, un);                                                                                       \
  }
#pragma unroll
        for (int q = 0; q < C8W; ++q) {
          float pp[8];
          TAOT_ROW_SUMS(q, pp)
          const float y = reduce8(pp, lane);  // all lanes take part
          TAOT_ROW_FINISH(q, y)
        }
#undef TAOT_ROW_FINISH
#undef TAOT_ROW_SUMS
        // outside [kLo, kHi], negative, infinite or NaN: this wave's rows are
        // updated exactly, then the iteration continues with its column half-step
        const bool fail = !(lo >= __float_as_uint(kLo) && hi <= __float_as_uint(kHi));
        if (__ballot(fail) != 0) {
          row_update = true;
          skip_row = true;
          break;
        }
      }
      skip_row = false;
      // ---- column half-step: v_c = d_c / sum_i u_i Kt_ic -------------------------------
      // this wave's row scalings reach its lanes through LDS (two broadcast
      // 16-byte loads per 8 rows; a wave's LDS accesses run in order)
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      // two partial sums per column (even and odd rows of each chunk), so
      // that 2 CPL independent FMA chains interleave
      float x[CPL], x2[CPL];
#pragma unroll
      for (int c = 0; c < CPL; ++c) x[c] = x2[c] = 0.f;
      // the loads of chunk q + 1 are issued before chunk q's FMAs
      float4 ua = *reinterpret_cast<const float4*>(ul + rb);
      float4 ub = *reinterpret_cast<const float4*>(ul + rb + 4);
#pragma unroll
      for (int q = 0; q < C8W; ++q) {
        float4 na = ua, nb = ub;
        if (q + 1 < C8W) {
          na = *reinterpret_cast<const float4*>(ul + rb + 8 * (q + 1));
          nb = *reinterpret_cast<const float4*>(ul + rb + 8 * (q + 1) + 4);
        }
        const float us[8] = {ua.x, ua.y, ua.z, ua.w, ub.x, ub.y, ub.z, ub.w};
#pragma unroll
        for (int r = 0; r < 8; r += 2)
#pragma unroll
          for (int c = 0; c < CPL; ++c) {
            x[c] = __builtin_fmaf(us[r], K[8 * q + r][c], x[c]);
            x2[c] = __builtin_fmaf(us[r + 1], K[8 * q + r + 1][c], x2[c]);
          }
        ua = na;
        ub = nb;
      }
#pragma unroll
      for (int c = 0; c < CPL; ++c) x[c] = x[c] + x2[c];
      if constexpr (NW > 1) {
        float* xs = xbuf + (size_t)((it & 1) * NW + wv) * CPL * kWave;
#pragma unroll
        for (int c = 0; c < CPL; ++c) xs[c * kWave + lane] = x[c];
        psync<NW>();
        const float* x0 = xbuf + (size_t)(it & 1) * NW * CPL * kWave;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          float sx = x0[c * kWave + lane];
#pragma unroll
          for (int w = 1; w < NW; ++w) sx = sx + x0[(w * CPL + c) * kWave + lane];
          x[c] = sx;
        }
      }
      // padding columns (all-zero Kt) divide by 1 and count as 1 in the range test
      float sB[CPL];
      demands(sB);
      uint32_t clo = 0xFFFFFFFFu, chi = 0u;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const float vn = sB[c] * frcp(CV(c) ? x[c] : 1.f);
        const uint32_t bits = __float_as_uint(CV(c) ? vn : 1.f);
        clo = bits < clo ? bits : clo;
        chi = bits > chi ? bits : chi;
        v[c] = vn;
      }
      // the same decision on every wave
      col_fail = __ballot(!(clo >= __float_as_uint(kLo) && chi <= __float_as_uint(kHi))) != 0;
      done = it == p.iters;
      if (!done) ++it;
      if (col_fail || done) break;
    }
    if (col_fail) {
      // exact log-domain update of every column, absorbed into G (online LSE
      // over all rows, whose scalings every wave has stored in ul); Kt is
      // rebuilt at the top of the loop, or below after the last iteration
      psync<NW>();
      float mx[CPL], sum[CPL];
#pragma unroll
      for (int c = 0; c < CPL; ++c) { mx[c] = -INFINITY; sum[c] = 0.f; }
      for (int32_t i = 0; i < nh; ++i) {
        const float fi = Fl[i] + flog2(ul[i]);
        const float* crow = Cb + (int64_t)hidx[i] * R;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          if (CV(c)) {
            const float t = fi - crow[CJ(c)] * kappa;
            const float m2 = fmaxf(mx[c], t);
            sum[c] = sum[c] * fexp2(mx[c] - m2) + fexp2(t - m2);
            mx[c] = m2;
          }
        }
      }
      float sB[CPL];
      demands(sB);
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        GL(c) = CV(c) ? flog2(sB[c]) - (mx[c] + flog2(sum[c])) : 0.f;
        v[c] = CV(c) ? 1.f : 0.f;
      }
      psync<NW>();  // every wave has read ul and F
      if (done) {
        build(false);
        break;
      }
      continue;
    }
    if (done) break;
  }

  // ---- plan, column cap, outputs -------------------------------------------------
  psync<NW>();  // the row scalings of every wave are in ul
  const bool colcap = !(p.flags & TAOT_SK_NO_COLCAP);
  float fac[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) fac[c] = 1.f;
  if (colcap) {
    float cs[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) cs[c] = 0.f;
#pragma unroll
    for (int i = 0; i < MW; ++i) {
      const float ui = ul[rb + i];
#pragma unroll
      for (int c = 0; c < CPL; ++c) cs[c] += ui * K[i][c] * v[c];
    }
    if constexpr (NW > 1) {
      // the iteration loop's last exchange used parity iters & 1
      float* xs = xbuf + (size_t)(((p.iters + 1) & 1) * NW + wv) * CPL * kWave;
#pragma unroll
      for (int c = 0; c < CPL; ++c) xs[c * kWave + lane] = cs[c];
      psync<NW>();
      const float* c0 = xbuf + (size_t)((p.iters + 1) & 1) * NW * CPL * kWave;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        float s = c0[c * kWave + lane];
#pragma unroll
        for (int w = 1; w < NW; ++w) s = s + c0[(w * CPL + c) * kWave + lane];
        cs[c] = s;
      }
    }
    float sB[CPL];
    demands(sB);
#pragma unroll
    for (int c = 0; c < CPL; ++c) fac[c] = CV(c) ? fminf(1.f, sB[c] / (cs[c] + 1e-12f)) : 1.f;
  }
  if (p.T) {
    float* Tb = p.T + pb * R * R;
    for (int32_t i = wv; i < R; i += NW) {
      const bool hot = hpos[i] >= 0;
      for (int32_t j = lane; j < R; j += kWave)
        if (!hot || cpos[j] < 0) Tb[(int64_t)i * R + j] = 0.f;
    }
#pragma unroll
    for (int i = 0; i < MW; ++i) {
      const int gi = rb + i;
      if (gi < nh) {
        const float ui = ul[gi];
        float* trow = Tb + (int64_t)hidx[gi] * R;
#pragma unroll
        for (int c = 0; c < CPL; ++c)
          if (CV(c)) trow[CJ(c)] = ui * K[i][c] * (v[c] * fac[c]);
      }
    }
  }
  if (wv == 0) {
    const float to_nat = p.eps * kLn2;
    for (int32_t i = lane; i < R; i += kWave) {
      const int32_t ih = hpos[i];
      if (p.f) p.f[pb * R + i] = ih >= 0 ? (Fl[ih] + flog2(ul[ih])) * to_nat : -INFINITY;
      if (p.g && cpos[i] < 0) p.g[pb * R + i] = -INFINITY;
    }
    if (p.g) {
#pragma unroll
      for (int c = 0; c < CPL; ++c)
        if (CV(c)) p.g[pb * R + CJ(c)] = (GL(c) + flog2(v[c])) * to_nat;
    }
    if (lane == 0 && p.status) p.status[pb] = 0u;
  }
#undef UST
#undef GL
#undef RV
#undef CJ
#undef CV
}

// ---------------------------------------------------------------------------
// One-wave layout with the columns folded over the two half-waves.  Lane l
// sits in half h = l >> 5 at column lane cl = l & 31 and owns compact columns
// cl, cl + 32, ... (CPL of them, so the block is padded to 32-column rather
// than 64-column steps); chunk q of 8 rows keeps rows 8q .. 8q+3 in half 0
// and 8q+4 .. 8q+7 in half 1, four Kt values per column.
//   row half-step:    per-lane partial sums of the half's 4 rows, then the
//                     transposed butterfly over the 32 lanes of each half
//                     (permlane16 swap, then DPP) leaves the total of row
//                     8q + (l >> 3) in lane l, as in the full-wave layout.
//   column half-step: partial sums over the half's rows; one permlane32 swap
//                     and an add per pair of columns (c, c + P) leave the
//                     totals of column c in half 0 and of column c + P in
//                     half 1, each half derives those scalings, and a second
//                     swap hands every lane both.
// Against the full-wave layout this drops one swap level from every row
// chunk (the halves' column partials meet once per iteration instead) and
// pads the columns less.

// Sums 4 per-lane values over the 32 lanes of each half-wave; lane l ends
// with the total of value (l >> 3) & 3 of its half.  The steps pair lanes
// l ^ 16 (permlane16 swap), l <-> 15 - l (row_mirror), l <-> l ^ 7
// (row_half_mirror), l ^ 2 and l ^ 1 (quad_perm).
__device__ __forceinline__ float reduce4(float (&p)[4], int lane) {
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
// Sums 8 per-lane values over the 32 lanes of each half-wave; lane l ends
// with the total of value 4 b4 + 2 b2 + b3 of its half (bk = bit k of l).
// The steps pair lanes l ^ 16 (permlane16 swap: values 0-3 stay in the lower
// row, 4-7 go to the upper), l <-> 15 - l (row_mirror, two independent
// chains), l <-> 7 - l (row_half_mirror), l ^ 2 and l ^ 1 (quad_perm).
__device__ __forceinline__ float reduce8h(float (&p)[8], int lane) {
#pragma unroll
  for (int k = 0; k < 4; ++k) { swap16(p[k], p[k + 4]); p[k] = p[k] + p[k + 4]; }
  const bool b3 = lane & 8, b2 = lane & 4;
  const float y0 = (b3 ? p[1] : p[0]) + dpp<0x140>(b3 ? p[0] : p[1]);  // value 4 b4 + b3
  const float y1 = (b3 ? p[3] : p[2]) + dpp<0x140>(b3 ? p[2] : p[3]);  // value 4 b4 + 2 + b3
  float z = (b2 ? y1 : y0) + dpp<0x141>(b2 ? y0 : y1);
  z = z + dpp<0x4E>(z);  // quad_perm [2,3,0,1]
  z = z + dpp<0xB1>(z);  // quad_perm [1,0,3,2]
  return z;
}
// Max and sum over the 32 lanes of each half-wave (bitwise the same in every
// lane of the half).
__device__ __forceinline__ float half_max(float x) {
  x = fmaxf(x, dpp<0xB1>(x));
  x = fmaxf(x, dpp<0x4E>(x));
  x = fmaxf(x, dpp<0x141>(x));
  x = fmaxf(x, dpp<0x140>(x));
  float y = x;
  swap16(x, y);
  return fmaxf(x, y);
}
__device__ __forceinline__ float half_sum(float x) {
  x = x + dpp<0xB1>(x);
  x = x + dpp<0x4E>(x);
  x = x + dpp<0x141>(x);
  x = x + dpp<0x140>(x);
  float y = x;
  swap16(x, y);
  return x + y;
}
// Both halves' values of v: a gets half 0's, b half 1's, in every lane.
__device__ __forceinline__ void halves_both(float v, float& a, float& b) {
  a = v;
  b = v;
  swap32(a, b);
}

// Chunks of 8 rows the folded layout holds for CPL columns per lane: 8 up to
// 128 columns, 6 beyond (the two-wave kernel runs a problem of more than 128
// columns on one wave only up to 6 chunks), at most 192 Kt registers.
__host__ __device__ constexpr int half_max_c8(int cpl) { return cpl <= 4 ? 8 : 6; }

// Iterations and outputs of one problem of c8 row chunks on this wave alone,
// in the folded layout; the caller has filled sAl and the first-update
// potentials Fl.  Gc [256] holds the column potentials by compact column, Sl
// [64][4] the demands of each lane's folded columns.
template <int CPL>
__device__ __forceinline__ void half_solve(const SkParams& p, int64_t pb, int32_t nh, int32_t nc, int c8,
                                           const int32_t* cpos, const int32_t* hpos, const int32_t* cidx,
                                           const int32_t* hidx, const float* sAl, float* Fl, float* ul, float* Gc,
                                           float* Sl, float kappa) {
  constexpr int MC = half_max_c8(CPL);  // chunks the registers hold; chunks q >= c8 are skipped
  constexpr int P = (CPL + 1) / 2;      // folded column pairs (c, c + P)
  const int lane = threadIdx.x & (kWave - 1);
  const int h = lane >> 5, cl = lane & 31;
  const int32_t R = p.R;
  const float* bd = p.b + pb * R;
  const float* Cb = p.C + pb * p.C_stride;
#define HV(c) (cl + 32 * (c) < nc)                 // column c of the lane exists
#define HJ(c) (HV(c) ? cidx[cl + 32 * (c)] : 0)   // its rank
#define FV(c) ((c) + P * h < CPL && cl + 32 * ((c) + P * h) < nc)  // folded column c of the lane exists
#define RV(q) (8 * (q) + (lane >> 3) < nh)        // the row the lane holds after reduce4
#define HR(q, r) (8 * (q) + 4 * h + (r))           // row r of chunk q in the lane's half
#define GL(c) Gc[cl + 32 * (c)]
  float* Sw = Sl + lane * 4;

  float K[4 * MC][CPL];
  float v[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    v[c] = HV(c) ? 1.f : 0.f;
    GL(c) = 0.f;  // both halves store the same value
  }
  // padding columns take demand 1, and padding rows supply 1 below, so that
  // their scalings come out as exactly 1 (in range, and Kt is 0 there)
#pragma unroll
  for (int c = 0; c < P; ++c) Sw[c] = FV(c) ? bd[cidx[cl + 32 * (c + P * h)]] : 1.f;
  auto demands = [&](float (&sB)[P]) {
#pragma unroll
    for (int c = 0; c < P; ++c) sB[c] = Sw[c];
  };
  // Kt of the lane's rows from the potentials (after the exact log-domain
  // update of each row's potential when row_update is set).  Rows past nh
  // take the cost row of row 0 and a zero Kt.
  auto build = [&](bool row_update) {
#pragma unroll
    for (int q = 0; q < MC; ++q) {
      if (q >= c8) break;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int gi = HR(q, r);
        const bool rv = gi < nh;
        const int gs = rv ? gi : 0;
        const float* crow = Cb + (int64_t)hidx[gs] * R;
        float cc[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) cc[c] = HV(c) ? crow[HJ(c)] * kappa : 0.f;
        float fi;
        if (row_update) {
          float t[CPL];
          float mx = -INFINITY;
#pragma unroll
          for (int c = 0; c < CPL; ++c) {
            t[c] = HV(c) ? (GL(c) + flog2(v[c])) - cc[c] : -INFINITY;
            mx = fmaxf(mx, t[c]);
          }
          mx = half_max(mx);
          float sum = 0.f;
#pragma unroll
          for (int c = 0; c < CPL; ++c) sum += HV(c) ? fexp2(t[c] - mx) : 0.f;
          sum = half_sum(sum);
          fi = flog2(sAl[gs]) - (mx + flog2(sum));
          if (rv && cl == 0) Fl[gi] = fi;
        } else {
          fi = Fl[gs];
        }
#pragma unroll
        for (int c = 0; c < CPL; ++c) K[4 * q + r][c] = rv && HV(c) ? fexp2((fi + GL(c)) - cc[c]) : 0.f;
      }
    }
  };

#define UST(q, val) \
  if ((lane & 7) == 0) ul[8 * (q) + (lane >> 3)] = (val)
#pragma unroll
  for (int q = 0; q < MC; ++q)
    if (q < c8) UST(q, RV(q) ? 1.f : 0.f);
  // Row half-steps take chunks in pairs (q, q + 1): reduce8h leaves the total
  // of row PR(q) in lane l; an odd last chunk goes through reduce4.
#define PR(q) (8 * ((q) + ((lane >> 4) & 1)) + 4 * h + 2 * ((lane >> 2) & 1) + ((lane >> 3) & 1))
  float sAp[MC / 2];
#pragma unroll
  for (int q = 0; q < MC; q += 2) sAp[q / 2] = PR(q) < nh ? sAl[PR(q)] : 1.f;
  const int qt = c8 - 1;  // the odd last chunk, when c8 is odd
  const float sAt = (c8 & 1) && RV(qt) ? sAl[8 * qt + (lane >> 3)] : 1.f;

  int32_t it = 1;
  bool skip_row = true;
  bool row_update = false;
  for (;;) {
    build(row_update);
    if (row_update) {
#pragma unroll
      for (int q = 0; q < MC; ++q)
        if (q < c8) UST(q, RV(q) ? 1.f : 0.f);
      row_update = false;
    }
    bool done = false, col_fail = false;
    for (;;) {
      if (!skip_row) {
        // ---- row half-step: u_i = s~_i / sum_c Kt_ic v_c ----------------------------
        uint32_t lo = 0xFFFFFFFFu, hi = 0u;
#pragma unroll
        for (int q = 0; q < MC; q += 2) {
          if (q >= c8) break;
          if (q + 1 < c8) {
            float pp[8];
#pragma unroll
            for (int r = 0; r < 8; ++r) {
              float acc = K[4 * q + r][0] * v[0];
#pragma unroll
              for (int c = 1; c < CPL; ++c) acc = __builtin_fmaf(K[4 * q + r][c], v[c], acc);
              pp[r] = acc;
            }
            // The reduction and the scaling are one dependent chain (each step
            // waits for the last): the wave takes a raised issue priority for
            // it, so that the SIMD's other wave, mostly in its FMA stretches,
            // fills the gaps instead of delaying the chain.
            __builtin_amdgcn_s_setprio(2);
            const float y = reduce8h(pp, lane);  // all lanes take part
            const float un = sAp[q / 2] * frcp(PR(q) < nh ? y : 1.f);
            const uint32_t bits = __float_as_uint(un);
            lo = bits < lo ? bits : lo;
            hi = bits > hi ? bits : hi;
            if ((lane & 3) == 0) ul[PR(q)] = un;
            __builtin_amdgcn_s_setprio(0);
          } else {
            float pp[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              float acc = K[4 * q + r][0] * v[0];
#pragma unroll
              for (int c = 1; c < CPL; ++c) acc = __builtin_fmaf(K[4 * q + r][c], v[c], acc);
              pp[r] = acc;
            }
            __builtin_amdgcn_s_setprio(2);
            const float y = reduce4(pp, lane);
            const float un = sAt * frcp(RV(q) ? y : 1.f);
            const uint32_t bits = __float_as_uint(un);
            lo = bits < lo ? bits : lo;
            hi = bits > hi ? bits : hi;
            UST(q, un);
            __builtin_amdgcn_s_setprio(0);
          }
        }
        const bool fail = !(lo >= __float_as_uint(kLo) && hi <= __float_as_uint(kHi));
        if (__ballot(fail) != 0) {
          row_update = true;
          skip_row = true;
          break;
        }
      }
      skip_row = false;
      // ---- column half-step: v_c = d_c / sum_i u_i Kt_ic --------------------------------
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      // with fewer than 4 columns per lane two partial sums per column (rows
      // 4q, 4q+2 and 4q+1, 4q+3) keep enough independent FMA chains in
      // flight; with 4 or more the columns alone do
      constexpr bool two = CPL < 4;
      float x[CPL], x2[CPL];
#pragma unroll
      for (int c = 0; c < CPL; ++c) x[c] = x2[c] = 0.f;
      float4 ua = *reinterpret_cast<const float4*>(ul + 4 * h);
#pragma unroll
      for (int q = 0; q < MC; ++q) {
        if (q >= c8) break;
        float4 na = ua;  // the next chunk's scalings (past c8: unused)
        if (q + 1 < MC) na = *reinterpret_cast<const float4*>(ul + 8 * (q + 1) + 4 * h);
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          x[c] = __builtin_fmaf(ua.x, K[4 * q][c], x[c]);
          if constexpr (two) x2[c] = __builtin_fmaf(ua.y, K[4 * q + 1][c], x2[c]);
          else x[c] = __builtin_fmaf(ua.y, K[4 * q + 1][c], x[c]);
          x[c] = __builtin_fmaf(ua.z, K[4 * q + 2][c], x[c]);
          if constexpr (two) x2[c] = __builtin_fmaf(ua.w, K[4 * q + 3][c], x2[c]);
          else x[c] = __builtin_fmaf(ua.w, K[4 * q + 3][c], x[c]);
        }
        ua = na;
      }
      // fold: register c of half 0 gets column c, of half 1 column c + P
      float xf[P];
#pragma unroll
      for (int c = 0; c < P; ++c) {
        float a = two ? x[c] + x2[c] : x[c];
        float b = c + P < CPL ? (two ? x[c + P] + x2[c + P] : x[c + P]) : 0.f;
        swap32(a, b);
        xf[c] = a + b;
      }
      float sB[P];
      demands(sB);
      uint32_t clo = 0xFFFFFFFFu, chi = 0u;
#pragma unroll
      for (int c = 0; c < P; ++c) {
        const float vn = sB[c] * frcp(FV(c) ? xf[c] : 1.f);
        const uint32_t bits = __float_as_uint(vn);
        clo = bits < clo ? bits : clo;
        chi = bits > chi ? bits : chi;
        float a, b;
        halves_both(vn, a, b);
        v[c] = a;
        if (c + P < CPL) v[c + P] = b;
      }
      col_fail = __ballot(!(clo >= __float_as_uint(kLo) && chi <= __float_as_uint(kHi))) != 0;
      done = it == p.iters;
      if (!done) ++it;
      if (col_fail || done) break;
    }
    if (col_fail) {
      // exact log-domain update of every column, absorbed into G: half h
      // takes the folded columns c + P h whose scalings it derives (online
      // LSE over all rows), and every lane reads G back; Kt is rebuilt at
      // the top of the loop, or below after the last iteration
      psync<1>();
      float mx[P], sum[P];
#pragma unroll
      for (int c = 0; c < P; ++c) { mx[c] = -INFINITY; sum[c] = 0.f; }
      for (int32_t i = 0; i < nh; ++i) {
        const float fi = Fl[i] + flog2(ul[i]);
        const uint32_t rowoff = (uint32_t)hidx[i] * (uint32_t)R;
#pragma unroll
        for (int c = 0; c < P; ++c) {
          if (FV(c)) {
            const float t = fi - Cb[rowoff + (uint32_t)cidx[cl + 32 * (c + P * h)]] * kappa;
            const float m2 = fmaxf(mx[c], t);
            sum[c] = sum[c] * fexp2(mx[c] - m2) + fexp2(t - m2);
            mx[c] = m2;
          }
        }
      }
#pragma unroll
      for (int c = 0; c < P; ++c)
        if (FV(c)) Gc[cl + 32 * (c + P * h)] = flog2(Sw[c]) - (mx[c] + flog2(sum[c]));
#pragma unroll
      for (int c = 0; c < CPL; ++c) v[c] = HV(c) ? 1.f : 0.f;
      psync<1>();
      if (done) {
        build(false);
        break;
      }
      continue;
    }
    if (done) break;
  }

  // ---- plan, column cap, outputs -------------------------------------------------
  psync<1>();
  const bool colcap = !(p.flags & TAOT_SK_NO_COLCAP);
  float fac[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) fac[c] = 1.f;
  if (colcap) {
    float cs[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) cs[c] = 0.f;
#pragma unroll
    for (int q = 0; q < MC; ++q) {
      if (q >= c8) break;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float ui = ul[HR(q, r)];
#pragma unroll
        for (int c = 0; c < CPL; ++c) cs[c] += ui * K[4 * q + r][c] * v[c];
      }
    }
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      float a, b;
      halves_both(cs[c], a, b);
      const float tot = a + b;
      fac[c] = HV(c) ? fminf(1.f, bd[HJ(c)] / (tot + 1e-12f)) : 1.f;
    }
  }
  if (p.T) {
    float* Tb = p.T + pb * R * R;
    for (int32_t i = 0; i < R; ++i) {
      const bool hot = hpos[i] >= 0;
      for (int32_t j = lane; j < R; j += kWave)
        if (!hot || cpos[j] < 0) Tb[(int64_t)i * R + j] = 0.f;
    }
#pragma unroll
    for (int q = 0; q < MC; ++q) {
      if (q >= c8) break;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int gi = HR(q, r);
        if (gi < nh) {
          const float ui = ul[gi];
          float* trow = Tb + (int64_t)hidx[gi] * R;
#pragma unroll
          for (int c = 0; c < CPL; ++c)
            if (HV(c)) trow[HJ(c)] = ui * K[4 * q + r][c] * (v[c] * fac[c]);
        }
      }
    }
  }
  const float to_nat = p.eps * kLn2;
  for (int32_t i = lane; i < R; i += kWave) {
    const int32_t ih = hpos[i];
    if (p.f) p.f[pb * R + i] = ih >= 0 ? (Fl[ih] + flog2(ul[ih])) * to_nat : -INFINITY;
    if (p.g && cpos[i] < 0) p.g[pb * R + i] = -INFINITY;
  }
  if (p.g && h == 0) {
#pragma unroll
    for (int c = 0; c < CPL; ++c)
      if (HV(c)) p.g[pb * R + HJ(c)] = (GL(c) + flog2(v[c])) * to_nat;
  }
  if (lane == 0 && p.status) p.status[pb] = 0u;
#undef UST
#undef PR
#undef GL
#undef HR
#undef RV
#undef FV
#undef HJ
#undef HV
}

// The solver instance of wave wv (uniform over the wave).
template <int CPL, int C8W, int NW>
__device__ __forceinline__ void solve_on_wave(int wv, const SkParams& p, int64_t pb, int32_t nh, int32_t nc,
                                              const int32_t* cpos, const int32_t* hpos, const int32_t* cidx,
                                              const int32_t* hidx, const float* sAl, float* Fl, float* ul,
                                              float* Gall, float* Sall, float* xbuf, float kappa) {
  if constexpr (NW == 1) {
    wave_solve<CPL, C8W, 1, 0>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, kappa);
  } else if constexpr (NW == 2) {
    if (wv == 0) wave_solve<CPL, C8W, 2, 0>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, kappa);
    else wave_solve<CPL, C8W, 2, 1>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, kappa);
  } else {
    switch (wv) {
      case 0: wave_solve<CPL, C8W, 4, 0>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, kappa); break;
      case 1: wave_solve<CPL, C8W, 4, 1>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, kappa); break;
      case 2: wave_solve<CPL, C8W, 4, 2>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, kappa); break;
      default: wave_solve<CPL, C8W, 4, 3>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, kappa); break;
    }
  }
}

// One problem on NW waves (NW = 1: this wave alone, beside other one-wave
// problems of the workgroup; NW = W: the whole workgroup of the W-wave kernel).
template <int NW, int W>
__device__ __forceinline__ void wave_problem(const SkParams& p, int64_t pb, int32_t* wl) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = NW == 1 ? 0 : __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);  // uniform
  const int32_t R = p.R;
  // float arrays first: ul is read 16 bytes at a time
  float* sAl = reinterpret_cast<float*>(wl);  // [64] scaled supply
  float* Fl = sAl + 64;                       // [64] absorbed row potentials (log2 units)
  float* ul = Fl + 64;                        // [64] row scalings
  float* Gall = ul + 64;                      // [NW][4][64] column potentials
  float* Sall = Gall + NW * 4 * kWave;        // [NW][64][4] column demands
  float* xbuf = Sall + NW * 4 * kWave;        // [2][NW][4][64] column exchange (NW > 1)
  int32_t* iw = reinterpret_cast<int32_t*>(reinterpret_cast<float*>(wl) + wave_lds_floats(NW));
  int32_t* cpos = iw + 4;        // [R] compact column, -1 if not cold (iw[0..3] unused)
  int32_t* hpos = cpos + R;      // [R] compact row of rank i, -1 if not hot
  int32_t* cidx = hpos + R;      // [256]
  int32_t* hidx = cidx + 256;    // [64]
  const float* a = p.a + pb * R;
  const float* bd = p.b + pb * R;
  const float* Cb = p.C + pb * p.C_stride;

  // ---- supports and mass (every wave, identical results) --------------------
  double sa = 0.0, sd = 0.0;
  int32_t nh = 0, nc = 0;
  for (int32_t base = 0; base < R; base += kWave) {
    const int32_t i = base + lane;
    const bool in = i < R;
    const float ai = in ? a[i] : 0.f, bi = in ? bd[i] : 0.f;
    sa += (double)ai;
    sd += (double)bi;
    const uint64_t hm = __ballot(in && ai > 0.f), cm = __ballot(in && bi > 0.f);
    const uint64_t below = (1ull << lane) - 1ull;
    const int32_t ph = nh + __popcll(hm & below), pc = nc + __popcll(cm & below);
    if (in) {
      hpos[i] = ai > 0.f ? ph : -1;
      cpos[i] = bi > 0.f ? pc : -1;
    }
    if (in && ai > 0.f && ph < 64) hidx[ph] = i;
    if (in && bi > 0.f && pc < 256) cidx[pc] = i;
    nh += __popcll(hm);
    nc += __popcll(cm);
  }
  sa = wave_sum_d(sa);
  sd = wave_sum_d(sd);
  double gamma = __shfl(sd, 0, kWave) / fmax(__shfl(sa, 0, kWave), kEps0);
  gamma = gamma < 1.0 ? gamma : 1.0;
  sAl[lane] = lane < nh ? (float)(gamma * (double)a[hidx[lane]]) : 0.f;  // zero padding to 64 rows
  psync<NW>();
  const float kappa = kLog2e / p.eps;

  // ---- first row update over all R columns (v = 1): F_i = log2 s~_i - LSE2_j(-C'_ij),
  // rows dealt out over the waves (the class prepass has left problems with
  // a non-finite cost to the LDS or streamed kernel)
  for (int32_t i = wv; i < nh; i += NW) {
    const float* crow = Cb + (int64_t)hidx[i] * R;
    float mx = -INFINITY;
    for (int32_t j = lane; j < R; j += kWave) mx = fmaxf(mx, -crow[j] * kappa);
    mx = lanes_max(mx);
    float sum = 0.f;
    for (int32_t j = lane; j < R; j += kWave) sum += fexp2(-crow[j] * kappa - mx);
    sum = lanes_sum(sum);
    if (lane == 0) Fl[i] = flog2(sAl[i]) - (mx + flog2(sum));
  }
  psync<NW>();
  if constexpr (NW == 1 && W == 2) {
    // one wave alone: the folded layout (every single class of the two-wave
    // kernel fits it)
    const int cph = (nc + 31) / 32, c8 = (nh + 7) / 8;
    switch (cph) {
#define TAOT_HALF_CASE(CPL_)                                                                          \
  case CPL_:                                                                                          \
    if (c8 >= 1 && c8 <= half_max_c8(CPL_)) {                                                         \
      half_solve<CPL_>(p, pb, nh, nc, c8, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, kappa);    \
      return;                                                                                         \
    }                                                                                                 \
    break;
      TAOT_HALF_CASE(1) TAOT_HALF_CASE(2) TAOT_HALF_CASE(3) TAOT_HALF_CASE(4)
      TAOT_HALF_CASE(5) TAOT_HALF_CASE(6) TAOT_HALF_CASE(7) TAOT_HALF_CASE(8)
#undef TAOT_HALF_CASE
      default: break;
    }
  } else {
    const int cpl = nc <= 64 ? 1 : nc <= 128 ? 2 : 4;
    const int c8w = ((nh + 7) / 8 + NW - 1) / NW;
    switch (cpl * 16 + c8w) {
#define TAOT_WAVE_CASE(CPL_, C8W_)                                                                    \
  case CPL_ * 16 + C8W_:                                                                              \
    if constexpr (shape_ok(W, NW, CPL_, C8W_))                                                        \
      solve_on_wave<CPL_, C8W_, NW>(wv, p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, \
                                    kappa);                                                           \
    break;
#define TAOT_WAVE_CPL(CPL_)                                                                           \
  TAOT_WAVE_CASE(CPL_, 1) TAOT_WAVE_CASE(CPL_, 2) TAOT_WAVE_CASE(CPL_, 3) TAOT_WAVE_CASE(CPL_, 4)      \
  TAOT_WAVE_CASE(CPL_, 5) TAOT_WAVE_CASE(CPL_, 6) TAOT_WAVE_CASE(CPL_, 7) TAOT_WAVE_CASE(CPL_, 8)
      TAOT_WAVE_CPL(1) TAOT_WAVE_CPL(2) TAOT_WAVE_CPL(4)
#undef TAOT_WAVE_CPL
#undef TAOT_WAVE_CASE
      default: break;
    }
  }
}

// The register problems of a batch on workgroups of G waves (G = W, or G = 8
// for the two-wave shapes): item k < n_multi is multi[k] on waves 0 .. W-1
// (any further waves end at once, and a barrier only waits for the waves that
// have not ended); item n_multi + g holds G single problems, one per wave,
// each wave with its own LDS slice.
//
// Single group g pairs the heavier half of the list (dealt from its front)
// with the lighter half (from its back), G / 2 problems each.  With G = 8 the
// group is the whole compute unit (eight 256-VGPR waves, two per SIMD), and
// the waves that share a SIMD share its issue slots: each wave reads its SIMD
// from the HW_ID register, and the k-th heaviest problem of the group goes to
// the first wave of the k-th SIMD, the k-th lightest to its second wave, so
// that every SIMD carries about the same work.  Any placement still gives
// every wave one distinct slot (slots ordered by rank within the SIMD, then
// by SIMD).
template <int W, int G>
__global__ void __launch_bounds__(G * kWave, W == 4 ? 4 : 2)
sinkhorn_reg_kernel(SkParams p, const int32_t* __restrict__ multi, const int32_t* __restrict__ single,
                    const int32_t* __restrict__ counts) {
  extern __shared__ __attribute__((aligned(16))) int32_t wl[];
  __shared__ int32_t simd_of[G];
  const int32_t n_multi = counts[0], n_single = counts[1];
  const int32_t k = blockIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if (k < n_multi) {
    if (w < W) wave_problem<W, W>(p, multi[k], wl);
    return;
  }
  const int64_t g = k - n_multi, F = ((int64_t)n_single + 1) / 2;
  if (g * (G / 2) >= F) return;  // past the last group (uniform over the workgroup)
  int slot = w;
  if constexpr (G > W) {
    // HW_ID bits 5:4 hold the SIMD of the wave
    const int simd = (int)__builtin_amdgcn_s_getreg((1 << 11) | (4 << 6) | 4);
    if ((threadIdx.x & (kWave - 1)) == 0) simd_of[w] = simd;
    __syncthreads();
    auto rank = [&](int u) {
      int r = 0;
      for (int t = 0; t < u; ++t) r += simd_of[t] == simd_of[u];
      return r;
    };
    const int mr = rank(w);
    int pos = 0;
    for (int u = 0; u < G; ++u) {
      const int ru = rank(u);
      pos += ru < mr || (ru == mr && simd_of[u] < simd);
    }
    slot = __builtin_amdgcn_readfirstlane(pos);
  }
  const bool front = slot < G / 2;
  const int kk = front ? slot : slot - G / 2;
  const int64_t j = front ? g * (G / 2) + kk : (int64_t)n_single - 1 - (g * (G / 2) + kk);
  if (front ? j < F : (j >= F && j < n_single))
    wave_problem<1, W>(p, single[j], wl + (size_t)w * (single_lds_bytes(p.R) / 4));
}

template <int W, int G>
taot_status launch_reg_kernel(const SkParams& p, const int32_t* multi, const int32_t* single, const int32_t* counts,
                              hipStream_t stream) {
  const size_t lds = std::max(wave_lds_bytes(p.R, W), (size_t)G * single_lds_bytes(p.R));
  if (lds > 65536 && hipFuncSetAttribute((const void*)sinkhorn_reg_kernel<W, G>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return TAOT_ERR_LAUNCH;
  // one workgroup per item at most: B is an upper bound on the items
  hipLaunchKernelGGL((sinkhorn_reg_kernel<W, G>), dim3((unsigned)p.B), dim3(G * kWave), lds, stream, p, multi,
                     single, counts);
  return hipGetLastError() == hipSuccess ? TAOT_OK : TAOT_ERR_LAUNCH;
}

}  // namespace
}  // namespace taot
