// DWT of the cached prompt keys (eqs. 5-6) and the skim: perception weights
// of the query block over the level-J approximation (eq. 7), their column
// sums W (eq. 8) and the top-S coarse regions (eq. 9).
//
// Layout: one unit = one (batch, head) pair; K is [U][L][D] with channels
// contiguous.  The DWT runs along the sequence independently per channel.
//
//  * Haar in the fused path: the level-J approximation of block j is
//    2^{-J/2} times the sum of its 2^J rows (the orthonormal pyramid
//    collapses to a block sum), so a wave streams rows with 16-byte loads,
//    accumulates in fp32 registers and finishes the block with cross-lane
//    butterflies.
//  * Daubechies-2 (and the staged transform that also returns details):
//    every lane owns two channels and runs the filter-bank cascade along the
//    sequence, level by level, with three samples of state per level; the
//    half-sample symmetric extension is applied per level at the true end.
//  * The skim epilogue multiplies the fp32 coefficient tile (in LDS) with
//    the query block on fp32 MFMA (v_mfma_f32_16x16x4_f32), then writes the
//    logits and per-tile row max / row sum of exponentials.  A per-unit
//    kernel merges the tiles' row statistics, forms W and selects.
#include <mutex>
#include <vector>

#include "wf_device.hpp"
#include "wf_kernels.hpp"
#include "wf_launch.hpp"

namespace wf {

struct Taps {
  float g[4];
  float h[4];
  float inv_norm;  // 2^{-J/2}, for the Haar block sum
};

struct F2 {
  float x, y;
};

__device__ __forceinline__ F2 load_pair(const bf16_t* p) {
  uint32_t w = *reinterpret_cast<const uint32_t*>(p);
  return F2{bf16_lo(w), bf16_hi(w)};
}
__device__ __forceinline__ F2 load_pair(const float* p) {
  u32x2 w = *reinterpret_cast<const u32x2*>(p);
  return F2{__uint_as_float(w[0]), __uint_as_float(w[1])};
}

// ------------------------------------------------------------ cascade

// Filter-bank cascade over one stream of rows for one channel pair.  Level j
// (1..J) consumes samples y^{j-1}[i] in increasing i and, after every odd i,
// emits y^j[n] = sum_m g_m y^{j-1}[2n+m] (and the detail with h), with
// n = (i - (M-1)) / 2.  Samples pushed before the stream's first aligned
// coefficient produce emissions with smaller indices, which sinks ignore.
template <int M, int J, bool DET>
struct Cascade {
  F2 s1[J + 1], s2[J + 1], s3[J + 1];  // y[i-1], y[i-2], y[i-3] per level
  float g0, g1, g2, g3, h0, h1, h2, h3;
  long L;
  bool symmetric;

  __device__ void init(const Taps& t, long L_, bool sym) {
    g0 = t.g[0]; g1 = t.g[1]; g2 = t.g[2]; g3 = t.g[3];
    h0 = t.h[0]; h1 = t.h[1]; h2 = t.h[2]; h3 = t.h[3];
    L = L_;
    symmetric = sym;
#pragma unroll
    for (int j = 0; j <= J; ++j) {
      s1[j] = F2{0.f, 0.f};
      s2[j] = F2{0.f, 0.f};
      s3[j] = F2{0.f, 0.f};
    }
  }

  template <int j, class Sink>
  __device__ __forceinline__ void feed(long i, F2 v, Sink& sink) {
    if (i & 1) {
      long n;
      F2 a, d;
      if constexpr (M == 2) {
        n = (i - 1) >> 1;
        a.x = g0 * s1[j].x + g1 * v.x;
        a.y = g0 * s1[j].y + g1 * v.y;
        if constexpr (DET) {
          d.x = h0 * s1[j].x + h1 * v.x;
          d.y = h0 * s1[j].y + h1 * v.y;
        }
      } else {
        n = (i - 3) >> 1;
        a.x = g0 * s3[j].x + g1 * s2[j].x + g2 * s1[j].x + g3 * v.x;
        a.y = g0 * s3[j].y + g1 * s2[j].y + g2 * s1[j].y + g3 * v.y;
        if constexpr (DET) {
          d.x = h0 * s3[j].x + h1 * s2[j].x + h2 * s1[j].x + h3 * v.x;
          d.y = h0 * s3[j].y + h1 * s2[j].y + h2 * s1[j].y + h3 * v.y;
        }
      }
      if constexpr (DET) sink.detail(j, n, d);
      if constexpr (j < J) {
        push<j + 1>(n, a, sink);
      } else {
        sink.approx(n, a);
      }
    }
    s3[j] = s2[j];
    s2[j] = s1[j];
    s1[j] = v;
  }

  // Pushes y^{j-1}[i].  After the last sample of a level (i = N - 1) the
  // symmetric mode continues with y[N] = y[N-1] and y[N+1] = y[N-2]
  // (half-sample symmetric extension); a loop keeps one copy of the deeper
  // levels' code.
  template <int j, class Sink>
  __device__ __forceinline__ void push(long i, F2 v, Sink& sink) {
    int reps = 1;
    const F2 prev = s1[j];
    if constexpr (M == 4) {
      if (symmetric && i == (L >> (j - 1)) - 1) reps = 3;
    }
#pragma unroll 1
    for (int r = 0; r < reps; ++r) {
      const F2 x = (r == 2) ? prev : v;
      feed<j>(i + r, x, sink);
    }
  }
};

// Rows a stream reads past its own 2^J-aligned range: level-J coefficient n
// of a 4-tap bank depends on rows 2^J n .. 2^J n + 3 (2^J - 1), so the last
// owned coefficient needs 2^{J+1} - 2 extra rows; a 2-tap bank needs none.
__host__ __device__ constexpr long cascade_halo(int M, int J) {
  return M == 4 ? (2L << J) - 2 : 0;
}

// Row t of the sequence a tile transforms: the unit's key row t, or on a
// refinement scale of the recursion row t of the gathered kept blocks
// (parent [npar] ids of 2^shift rows each; ids are clamped into the unit).
struct RowsIdentity {
  __device__ __forceinline__ long operator()(long t) const { return t; }
};
struct RowsGathered {
  const int32_t* par;
  int shift;
  long last;
  __device__ __forceinline__ long operator()(long t) const {
    const long r = ((long)par[t >> shift] << shift) | (t & ((1L << shift) - 1));
    return min(max(r, 0L), last);
  }
};

// Streams rows [t0, t_stop) of one unit into the cascade (periodic extension
// reads row t mod L), 16 loads in flight per lane.
template <int M, int J, bool DET, typename T, class Sink, class RowMap = RowsIdentity>
__device__ void run_stream(Cascade<M, J, DET>& cas, const T* Kunit, int D,
                           int cp, long t0, long t_stop, long L, Sink& sink,
                           const RowMap& map = RowMap{}) {
  constexpr int U = 16;
  for (long t = t0; t < t_stop; t += U) {
    F2 v[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      long tt = t + k;
      if (tt < t_stop) {
        long row = tt < L ? tt : tt % L;
        v[k] = load_pair(Kunit + map(row) * D + 2 * cp);
      } else {
        v[k] = F2{0.f, 0.f};
      }
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      if (t + k < t_stop) cas.template push<1>(t + k, v[k], sink);
    }
  }
}

struct GlobalSink {
  float* aout;     // approximation, unit base + 2 cp
  float* dout;     // details, unit base + 2 cp, nullable
  long n0, n1;     // level-J rows owned by the stream
  long L;
  int J, D;
  __device__ __forceinline__ void store2(float* p, F2 a) {
    *reinterpret_cast<float2*>(p) = make_float2(a.x, a.y);
  }
  __device__ __forceinline__ void approx(long n, F2 a) {
    if (n >= n0 && n < n1) store2(aout + n * D, a);
  }
  __device__ __forceinline__ void detail(int j, long n, F2 d) {
    const long lo = n0 << (J - j), hi = n1 << (J - j);
    if (dout && n >= lo && n < hi) {
      const long row = (L - (L >> (j - 1))) + n;  // D_1 rows come first
      store2(dout + row * D, d);
    }
  }
};

struct LdsSink {
  float* coef;  // tile base + 2 cp
  long nbase;   // coefficient index of tile row 0
  long n0, n1;  // rows owned by the stream
  int stride;
  __device__ __forceinline__ void approx(long n, F2 a) {
    if (n >= n0 && n < n1) {
      float* p = coef + (n - nbase) * stride;
      p[0] = a.x;
      p[1] = a.y;
    }
  }
  __device__ __forceinline__ void detail(int, long, F2) {}
};

// ------------------------------------------------------------ staged DWT

template <int M, int J, typename T>
__global__ __launch_bounds__(kBlock) void dwt_kernel(DwtArgs a, Taps taps) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lps = a.D / 2;             // lanes per stream
  const int spw = kWave / lps;         // streams per wave
  const int cp = lane % lps;
  const int sid = wave * spw + lane / lps;
  const int u = blockIdx.x / a.ntiles;
  const int tile = blockIdx.x % a.ntiles;
  const long n0 = ((long)tile * a.streams + sid) * a.cps;
  if (u >= a.U || n0 >= a.nJ) return;  // no barrier in this kernel
  const long n1 = min(n0 + (long)a.cps, (long)a.nJ);
  const T* Kunit = reinterpret_cast<const T*>(a.K) + (long)u * a.Ls * a.D;
  GlobalSink sink;
  sink.aout = a.approx + (long)u * a.nJ * a.D + 2 * cp;
  sink.dout = a.details ? a.details + (long)u * (a.L - a.nJ) * a.D + 2 * cp
                        : nullptr;
  sink.n0 = n0;
  sink.n1 = n1;
  sink.L = a.L;
  sink.J = J;
  sink.D = a.D;
  Cascade<M, J, true> cas;
  const bool sym = (M == 4) && a.boundary == 0;
  cas.init(taps, a.L, sym);
  const long t0 = n0 << J;
  long t_stop = (n1 << J) + cascade_halo(M, J);
  if (sym || M == 2) t_stop = min(t_stop, (long)a.L);
  run_stream<M, J, true, T>(cas, Kunit, a.D, cp, t0, t_stop, a.L, sink);
}

// ------------------------------------------------------------ skim tiles

// Haar level-J approximation of tile rows [n0, n0 + ncoef) into LDS.
// Coefficient n covers tokens bid(n) 2^J .. bid(n) 2^J + 2^J - 1.  A wave
// sums groups of G = max(2^J, RPL) rows (RPL rows per 16-byte wave load):
// one coefficient per group, or RPL / 2^J of them reduced across lanes.
// LOADS = G / RPL loads per group (8 stands for 8 or more); small groups
// are taken 8 / LOADS at a time so that a lane always has 8 loads in flight.
template <typename T, int D, int LOADS, class BlockId>
__device__ void haar_sum_tile_groups(const T* Kunit, long n0, int ncoef, int J,
                                     float inv_norm, float* coef, const BlockId& bid) {
  constexpr int CPL = 16 / sizeof(T);  // channels per lane (16-byte load)
  constexpr int LPR = D / CPL;         // lanes per row
  constexpr int RPL = kWave / LPR;     // rows per wave load
  constexpr int STRIDE = D + kCoefPad;
  constexpr int NW = kBlock / kWave;
  constexpr int GPI = LOADS >= 8 ? 1 : 8 / LOADS;  // groups per iteration
  constexpr int LPI = LOADS >= 8 ? 8 : LOADS;      // loads per group and batch
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rsub = lane / LPR, csub = lane % LPR;
  const int blk = 1 << J;
  const int G = blk > RPL ? blk : RPL;
  const int cpg = G / blk;                // coefficients per group
  const int red = blk < RPL ? blk : RPL;  // rows reduced across lanes
  const long rows = (long)ncoef << J;     // tile rows, in coefficient order
  const int ngroups = (int)((rows + G - 1) / G);
  const int nloads = LOADS >= 8 ? G / RPL : 1;  // batches of LPI loads per group
  for (int gb = wave; gb < ngroups; gb += NW * GPI) {
    float acc[GPI][CPL];
#pragma unroll
    for (int gi = 0; gi < GPI; ++gi)
#pragma unroll
      for (int e = 0; e < CPL; ++e) acc[gi][e] = 0.f;
    for (int i0 = 0; i0 < nloads; i0 += LPI) {
      u32x4 v[GPI][LPI];
#pragma unroll
      for (int gi = 0; gi < GPI; ++gi)
#pragma unroll
        for (int li = 0; li < LPI; ++li) {
          const int grp = gb + gi * NW;
          const long r = (long)grp * G + rsub + (long)(i0 + li) * RPL;
          if (grp < ngroups && r < rows) {
            const long t = ((long)bid(n0 + (r >> J)) << J) + (r & (blk - 1));
            v[gi][li] = *reinterpret_cast<const u32x4*>(Kunit + t * D + csub * CPL);
          } else {
            v[gi][li] = u32x4{0u, 0u, 0u, 0u};
          }
        }
#pragma unroll
      for (int gi = 0; gi < GPI; ++gi)
#pragma unroll
        for (int li = 0; li < LPI; ++li) {
          if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              acc[gi][2 * e] += bf16_lo(v[gi][li][e]);
              acc[gi][2 * e + 1] += bf16_hi(v[gi][li][e]);
            }
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[gi][e] += __uint_as_float(v[gi][li][e]);
          }
        }
    }
#pragma unroll
    for (int gi = 0; gi < GPI; ++gi) {
      // the red rows of a coefficient sit LPR, 2 LPR, ... lanes apart (LDS
      // permutes: with many waves resident their latency hides, where the
      // VALU lane swaps would take issue slots)
#pragma unroll
      for (int sh = 1; sh < red; sh <<= 1) {
#pragma unroll
        for (int e = 0; e < CPL; ++e) acc[gi][e] += __shfl_xor(acc[gi][e], LPR * sh);
      }
      const int grp = gb + gi * NW;
      if (grp < ngroups && rsub % red == 0) {
        const int c = grp * cpg + rsub / blk;
        if (c < ncoef) {
          float* dst = coef + c * STRIDE + csub * CPL;
#pragma unroll
          for (int e = 0; e < CPL; ++e) dst[e] = acc[gi][e] * inv_norm;
        }
      }
    }
  }
}

template <typename T, int D, class BlockId>
__device__ void haar_sum_tile(const T* Kunit, long n0, int ncoef, int J, float inv_norm,
                              float* coef, const BlockId& bid) {
  constexpr int RPL = kWave / (D / (16 / (int)sizeof(T)));
  const int blk = 1 << J;
  const int loads = (blk > RPL ? blk : RPL) / RPL;
  switch (loads) {
    case 1: haar_sum_tile_groups<T, D, 1>(Kunit, n0, ncoef, J, inv_norm, coef, bid); break;
    case 2: haar_sum_tile_groups<T, D, 2>(Kunit, n0, ncoef, J, inv_norm, coef, bid); break;
    case 4: haar_sum_tile_groups<T, D, 4>(Kunit, n0, ncoef, J, inv_norm, coef, bid); break;
    default: haar_sum_tile_groups<T, D, 8>(Kunit, n0, ncoef, J, inv_norm, coef, bid); break;
  }
}

// Cascade level-J approximation of tile rows [n0, n0 + ncoef) into LDS.
// The tile is split into one stream per half/whole wave.
template <int M, int J, typename T, int D, class RowMap>
__device__ void cascade_tile(const T* Kunit, long L, long n0, int ncoef,
                             int cpt, bool sym, const Taps& taps,
                             float* coef, const RowMap& map) {
  constexpr int LPS = D / 2;
  constexpr int SPW = kWave / LPS;
  constexpr int NSTREAM = (kBlock / kWave) * SPW;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int cp = lane % LPS;
  const int sid = wave * SPW + lane / LPS;
  const int cps = cpt / NSTREAM;
  const long s0 = n0 + (long)sid * cps;
  const long s1 = min(s0 + (long)cps, n0 + (long)ncoef);
  if (s0 >= s1) return;
  LdsSink sink;
  sink.coef = coef + 2 * cp;
  sink.nbase = n0;
  sink.n0 = s0;
  sink.n1 = s1;
  sink.stride = D + kCoefPad;
  Cascade<M, J, false> cas;
  cas.init(taps, L, sym);
  const long t0 = s0 << J;
  long t_stop = (s1 << J) + cascade_halo(M, J);
  if (sym || M == 2) t_stop = min(t_stop, L);
  run_stream<M, J, false, T>(cas, Kunit, D, cp, t0, t_stop, L, sink, map);
}

// ------------------------------------------------------------ banded filter

// Away from the end of the sequence the level-J approximation of a 4-tap
// bank is one banded filter: A_J[n] = sum_m f_J[m] y0[2^J n + m] with
// f_1 = g and f_{j+1}[s] = sum_k g_k f_j[s - 2^j k] (length 3 (2^J - 1) + 1).
// With the symmetric extension the per-level extensions do not compose, so
// the filter is exact only while 2^J n + 3 (2^J - 1) < L; the periodic
// extension composes (even lengths), with rows read modulo L.
__host__ __device__ constexpr int band_len(int J) { return 3 * ((1 << J) - 1) + 1; }

// Rows a 16-byte wave load covers and whether the banded fill applies: every
// load must lie inside one 2^J-row block.
template <typename T, int D, int J>
struct BandShape {
  static constexpr int CPL = 16 / (int)sizeof(T);  // channels per lane
  static constexpr int LPR = D / CPL;              // lanes per row
  static constexpr int RPI = kWave / LPR;          // rows per load
  static constexpr bool ok = (1 << J) >= RPI;
};

// f_J into taps[0 .. 3 2^J) (zero past its length), built in LDS by the
// whole workgroup from the 4 low-pass taps; tmp is scratch of the same size.
template <int J>
__device__ void build_band_taps(const Taps& t, float* taps, float* tmp) {
  constexpr int N = 3 << J;
  float* cur = (J % 2 == 1) ? taps : tmp;  // f_1 lands where f_J ends up
  for (int i = threadIdx.x; i < N; i += kBlock) cur[i] = i < 4 ? t.g[i] : 0.f;
  __syncthreads();
  for (int j = 1; j < J; ++j) {
    float* nxt = cur == taps ? tmp : taps;
    const int step = 1 << j;
    for (int i = threadIdx.x; i < N; i += kBlock) {
      float v = 0.f;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int src = i - step * k;
        if (src >= 0) v += t.g[k] * cur[src];
      }
      nxt[i] = v;
    }
    __syncthreads();
    cur = nxt;
  }
}

// Sum of v over the lanes l ^ sh, sh = LPR .. 32 (the RPI rows of a load).
template <int LPR>
__device__ __forceinline__ float sum_rows(float v) {
  if constexpr (LPR <= 8)
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xf, 0xf, false));
  if constexpr (LPR <= 16) v = add_xor16(v);
  v = add_xor32(v);
  return v;
}

// Level-J approximation of coefficients [n0, n0 + ncoef) ∩ [0, n_end) into
// the LDS tile by the banded filter.  Wave w takes a contiguous run of the
// tile's coefficients and streams their rows once: at block b a lane adds
// its row's contribution to coefficients b, b - 1, b - 2 (taps o, o + 2^J,
// o + 2^(J+1) at offset o in the block); when block b + 1 starts,
// coefficient b - 2 is complete and its RPI row lanes are summed.
template <typename T, int D, int J, class RowMap>
__device__ void band_tile(const T* Kunit, long L, long n0, int ncoef, long n_end,
                          bool periodic, const float* taps, float* coef, const RowMap& map) {
  using BS = BandShape<T, D, J>;
  constexpr int CPL = BS::CPL, LPR = BS::LPR, RPI = BS::RPI;
  constexpr int BLK = 1 << J;
  constexpr int GPB = BLK / RPI;  // loads per block
  constexpr int BATCH = GPB < 8 ? GPB : 8;
  constexpr int STRIDE = D + kCoefPad;
  constexpr int NW = kBlock / kWave;
  static_assert(BS::ok, "a load must stay inside one block");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rsub = lane / LPR, csub = lane % LPR;
  const int per = (ncoef + NW - 1) / NW;
  const long c0 = n0 + (long)wave * per;
  const long c1 = min(min(c0 + (long)per, n0 + (long)ncoef), n_end);
  if (c0 >= c1) return;  // uniform per wave; no barrier follows inside
  float a0[CPL], a1[CPL], a2[CPL];  // coefficients b, b - 1, b - 2
#pragma unroll
  for (int e = 0; e < CPL; ++e) a0[e] = a1[e] = a2[e] = 0.f;
  auto flush = [&](long n) {
    float r[CPL];
#pragma unroll
    for (int e = 0; e < CPL; ++e) r[e] = sum_rows<LPR>(a2[e]);
    if (rsub == 0 && n >= c0 && n < c1) {
      float* dst = coef + (n - n0) * STRIDE + csub * CPL;
#pragma unroll
      for (int e = 0; e < CPL; e += 4)
        *reinterpret_cast<f32x4*>(dst + e) = f32x4{r[e], r[e + 1], r[e + 2], r[e + 3]};
    }
  };
  // batches of BATCH loads over blocks c0 .. c1 + 1
  constexpr int NBB = GPB / BATCH;  // batches per block
  const long nbt = (c1 + 2 - c0) * NBB;
  for (long bi = 0; bi < nbt; ++bi) {
    const long b = c0 + bi / NBB;
    const int g0 = (int)(bi % NBB) * BATCH;
    u32x4 v[BATCH];
#pragma unroll
    for (int gi = 0; gi < BATCH; ++gi) {
      const long r = b * BLK + (g0 + gi) * RPI + rsub;
      // past L: wrapped (periodic) or the last row with a zero tap
      const long row = r < L ? r : (periodic ? r % L : L - 1);
      v[gi] = *reinterpret_cast<const u32x4*>(Kunit + map(row) * D + csub * CPL);
    }
    if (g0 == 0 && b > c0) {
      flush(b - 3);
#pragma unroll
      for (int e = 0; e < CPL; ++e) {
        a2[e] = a1[e];
        a1[e] = a0[e];
        a0[e] = 0.f;
      }
    }
#pragma unroll
    for (int gi = 0; gi < BATCH; ++gi) {
      const int o = (g0 + gi) * RPI + rsub;
      const float t0 = taps[o], t1 = taps[o + BLK], t2 = taps[o + 2 * BLK];
      float x[CPL];
      if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x[2 * e] = bf16_lo(v[gi][e]);
          x[2 * e + 1] = bf16_hi(v[gi][e]);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = __uint_as_float(v[gi][e]);
      }
#pragma unroll
      for (int e = 0; e < CPL; ++e) {
        a0[e] = fmaf(t0, x[e], a0[e]);
        a1[e] = fmaf(t1, x[e], a1[e]);
        a2[e] = fmaf(t2, x[e], a2[e]);
      }
    }
  }
  flush(c1 - 1);
}

// The coefficients next to a symmetric end: coefficient nJ - 1 - m (m < 3)
// is sum_r E_m[r] y0[(nJ - 1 - m) 2^J + r], r < 2^J (m + 1).  The per-level
// extensions make E_m differ from f_J, but E_m depends only on m (lengths
// are multiples of 2^J), so the host builds the three filters once per J by
// pushing impulses through the extended cascade.  Filter m starts at
// 2^J m (m + 1) / 2.  The banded path with edges covers J <= kBandMaxJ.
constexpr int kBandMaxJ = 7;
struct EdgeTaps {
  float e[6 << kBandMaxJ];
};

// Edge coefficient n of the tile into LDS by the calling wave.
template <typename T, int D, int J, class RowMap>
__device__ void edge_coef(const T* Kunit, long n0, long n, long nJ, const float* edge,
                          float* coef, const RowMap& map) {
  using BS = BandShape<T, D, J>;
  constexpr int CPL = BS::CPL, LPR = BS::LPR, RPI = BS::RPI;
  constexpr int BLK = 1 << J;
  constexpr int STRIDE = D + kCoefPad;
  const int lane = threadIdx.x & 63;
  const int rsub = lane / LPR, csub = lane % LPR;
  const int m = (int)(nJ - 1 - n);
  const float* e = edge + BLK * (m * (m + 1) / 2);
  const int len = BLK * (m + 1);  // rows n 2^J .. L - 1
  float acc[CPL];
#pragma unroll
  for (int k = 0; k < CPL; ++k) acc[k] = 0.f;
  for (int r0 = 0; r0 < len; r0 += RPI) {
    const int rr = r0 + rsub;
    const u32x4 v = *reinterpret_cast<const u32x4*>(Kunit + map(n * BLK + rr) * D + csub * CPL);
    const float t = e[rr];
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        acc[2 * k] = fmaf(t, bf16_lo(v[k]), acc[2 * k]);
        acc[2 * k + 1] = fmaf(t, bf16_hi(v[k]), acc[2 * k + 1]);
      }
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[k] = fmaf(t, __uint_as_float(v[k]), acc[k]);
    }
  }
#pragma unroll
  for (int k = 0; k < CPL; ++k) acc[k] = sum_rows<LPR>(acc[k]);
  if (rsub == 0) {
    float* dst = coef + (n - n0) * STRIDE + csub * CPL;
#pragma unroll
    for (int k = 0; k < CPL; k += 4)
      *reinterpret_cast<f32x4*>(dst + k) = f32x4{acc[k], acc[k + 1], acc[k + 2], acc[k + 3]};
  }
}

// In place, every fp32 coefficient row of the tile becomes [hi x D][lo x D]
// bf16 in the same bytes: hi = bf16(c), lo = bf16(c - hi) (round to nearest
// even), so |c - hi - lo| <= 2^-17 |c|.  The whole workgroup reads, then
// writes (the halves overlap other threads' sources); it ends with a barrier.
template <int D>
__device__ void split_tile_bf16(float* coef, int ncoef) {
  constexpr int STRIDE = D + kCoefPad;
  constexpr int GPR = D / 8;  // 8-channel groups per row
  constexpr int MAXI = kMaxCoefTile * GPR / kBlock;
  uint32_t hi[MAXI][4], lo[MAXI][4];
#pragma unroll
  for (int k = 0; k < MAXI; ++k) {
    const int it = threadIdx.x + k * kBlock, row = it / GPR, grp = it % GPR;
    if (row < ncoef) {
      const float* src = coef + row * STRIDE + 8 * grp;
      const f32x4 v0 = *reinterpret_cast<const f32x4*>(src);
      const f32x4 v1 = *reinterpret_cast<const f32x4*>(src + 4);
      const float v[8] = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        hi[k][e] = pack_bf16x2(v[2 * e], v[2 * e + 1]);
        lo[k][e] = pack_bf16x2(v[2 * e] - bf16_lo(hi[k][e]), v[2 * e + 1] - bf16_hi(hi[k][e]));
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < MAXI; ++k) {
    const int it = threadIdx.x + k * kBlock, row = it / GPR, grp = it % GPR;
    if (row < ncoef) {
      unsigned char* dst = reinterpret_cast<unsigned char*>(coef + row * STRIDE);
      *reinterpret_cast<u32x4*>(dst + 16 * grp) = u32x4{hi[k][0], hi[k][1], hi[k][2], hi[k][3]};
      *reinterpret_cast<u32x4*>(dst + 2 * D + 16 * grp) = u32x4{lo[k][0], lo[k][1], lo[k][2], lo[k][3]};
    }
  }
  __syncthreads();
}

// logits[q][n0 + c] = scale * <Q_q, coef_c> for the tile, plus per-row max
// and sum of exp over the tile's columns.
template <typename T, int D>
__device__ void skim_epilogue(const SkimTileArgs& a, int u, int tile, long n0,
                              int ncoef, const float* coef) {
  constexpr int STRIDE = D + kCoefPad;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, col = lane & 15;
  const int nqb = (a.B + 15) / 16;
  const int ncb = (ncoef + 15) / 16;
  const T* Qunit = reinterpret_cast<const T*>(a.Q) + (long)u * a.B * D;
  for (int qb = wave; qb < nqb; qb += kBlock / kWave) {
    const int qrow = min(qb * 16 + col, a.B - 1);  // clamped query row
    f32x4 acc[kMaxCoefTile / 16];
    if constexpr (sizeof(T) == 2) {
      // bf16 queries are exact; the tile holds each coefficient row as
      // [hi x D][lo x D] bf16 (split_tile_bf16), so two bf16 products give
      // the fp32 dot product to within 2^-17 of each term.  A operand: query
      // row, channels 32 s + 8 g ..; B operand: the same channels of
      // coefficient 16 cb + col.
      u32x4 qa[D / 32];
#pragma unroll
      for (int s32 = 0; s32 < D / 32; ++s32)
        qa[s32] = *reinterpret_cast<const u32x4*>(Qunit + (long)qrow * D + 32 * s32 + 8 * g);
#pragma unroll
      for (int cb = 0; cb < kMaxCoefTile / 16; ++cb) {
        acc[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (cb < ncb) {
          const unsigned char* crow =
              reinterpret_cast<const unsigned char*>(coef + (cb * 16 + col) * STRIDE);
#pragma unroll
          for (int s32 = 0; s32 < D / 32; ++s32) {
            const u32x4 hi = *reinterpret_cast<const u32x4*>(crow + 2 * (32 * s32 + 8 * g));
            const u32x4 lo = *reinterpret_cast<const u32x4*>(crow + 2 * D + 2 * (32 * s32 + 8 * g));
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, qa[s32]), __builtin_bit_cast(bf16x8, hi), acc[cb], 0, 0, 0);
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, qa[s32]), __builtin_bit_cast(bf16x8, lo), acc[cb], 0, 0, 0);
          }
        }
      }
    } else {
      // A operand: query row, channels [g D/4, (g+1) D/4) (fp32 products)
      float qv[D / 4];
      const T* qsrc = Qunit + (long)qrow * D + g * (D / 4);
#pragma unroll
      for (int v = 0; v < D / 16; ++v) {
        f32x4 w = *reinterpret_cast<const f32x4*>(qsrc + 4 * v);
#pragma unroll
        for (int e = 0; e < 4; ++e) qv[4 * v + e] = w[e];
      }
#pragma unroll
      for (int cb = 0; cb < kMaxCoefTile / 16; ++cb) {
        acc[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (cb < ncb) {
          const float* crow = coef + (cb * 16 + col) * STRIDE + g * (D / 4);
#pragma unroll
          for (int s4 = 0; s4 < D / 16; ++s4) {
            f32x4 cv = *reinterpret_cast<const f32x4*>(crow + 4 * s4);
#pragma unroll
            for (int e = 0; e < 4; ++e)
              acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(qv[4 * s4 + e], cv[e], acc[cb], 0, 0, 0);
          }
        }
      }
    }
    // lane holds logit[q = 16 qb + 4 g + i][c = 16 cb + col]
    float m[4], z[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mx = -INFINITY;
#pragma unroll
      for (int cb = 0; cb < kMaxCoefTile / 16; ++cb) {
        const int c = cb * 16 + col;
        const bool ok = cb < ncb && c < ncoef;
        const float v = ok ? acc[cb][i] * a.scale : -INFINITY;
        acc[cb][i] = v;
        mx = fmaxf(mx, v);
      }
      m[i] = wave_max16(mx);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float s = 0.f;
#pragma unroll
      for (int cb = 0; cb < kMaxCoefTile / 16; ++cb) {
        const int c = cb * 16 + col;
        if (cb < ncb && c < ncoef) s += __expf(acc[cb][i] - m[i]);
      }
      s = wave_sum16(s);
      z[i] = s;
    }
    float* lg = a.logits + (long)u * a.B * a.nJ + n0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int q = qb * 16 + 4 * g + i;
      if (q < a.B) {
#pragma unroll
        for (int cb = 0; cb < kMaxCoefTile / 16; ++cb) {
          const int c = cb * 16 + col;
          if (cb < ncb && c < ncoef) lg[(long)q * a.nJ + c] = acc[cb][i];
        }
      }
    }
    if (col == 0) {
      float* st = a.stats + ((long)u * a.ntiles + tile) * 2 * a.B;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = qb * 16 + 4 * g + i;
        if (q < a.B) {
          st[q] = m[i];
          st[a.B + q] = z[i];
        }
      }
    }
  }
}

// Waves per SIMD a skim tile instance is compiled for.  The banded db2
// tiles at J = 6, 7 (d = 128, bf16) fit four workgroups per CU in 128 VGPRs
// without spills, so one round of workgroups covers the 32 tiles per unit of
// the 128K shape instead of a round and a third; other instances would
// spill under that bound and keep the default.
constexpr int skim_tile_waves(int src, int M, int J, int elem, int D) {
  return src == kCascade && M == 4 && elem == 2 && D == 128 && (J == 6 || J == 7) ? 4 : 1;
}

template <int SRC, int M, int J, typename T, int D>
__global__ __launch_bounds__(kBlock, skim_tile_waves(SRC, M, J, (int)sizeof(T), D)) void
skim_tile_kernel(SkimTileArgs a, Taps taps, EdgeTaps edge) {
  extern __shared__ float coef[];  // [cpt][D + kCoefPad], then the banded taps
  constexpr bool kBand = SRC == kCascade && M == 4 && BandShape<T, D, J>::ok && J <= kBandMaxJ;
  float* band = coef + a.cpt * (D + kCoefPad);  // [2][3 << J], then [6 << J] edge filters
  float* edge_lds = band + 2 * (3 << J);
  if constexpr (kBand) {
    for (int i = threadIdx.x; i < (6 << J); i += kBlock) edge_lds[i] = edge.e[i];
    build_band_taps<J>(taps, band, band + (3 << J));  // ends with a barrier
  }
  const int total = a.U * a.ntiles;
  for (int item = blockIdx.x; item < total; item += gridDim.x) {
    const int u = item / a.ntiles;
    const int tile = item % a.ntiles;
    const long n0 = (long)tile * a.cpt;
    const int ncoef = (int)min((long)a.cpt, (long)a.nJ - n0);
    if constexpr (SRC == kHaarSum) {
      const T* Kunit = reinterpret_cast<const T*>(a.K) + (long)u * a.Ls * D;
      if (a.parent) {
        // block ids are clamped into the unit: a bad id cannot leave K
        const int32_t* par = a.parent + (long)u * a.npar;
        const long last = ((long)a.L >> a.J) - 1;
        haar_sum_tile<T, D>(Kunit, n0, ncoef, a.J, taps.inv_norm, coef, [=](long n) {
          return min(max(2L * par[n >> 1] + (n & 1), 0L), last);
        });
      } else {
        haar_sum_tile<T, D>(Kunit, n0, ncoef, a.J, taps.inv_norm, coef,
                            [](long n) { return n; });
      }
    } else if constexpr (SRC == kCascade) {
      const T* Kunit = reinterpret_cast<const T*>(a.K) + (long)u * a.Ls * D;
      const bool sym = M == 4 && a.boundary == 0;
      // a.L rows: the filtered keys, or on a refinement scale of the
      // recursion the gathered kept blocks (eq. 11), read across their joins
      auto transform = [&](const auto& map) {
        if constexpr (kBand) {
          // interior coefficients by the banded filter, those whose window
          // reaches a symmetric end by the end filters (a wave each)
          const long nJf = (long)a.L >> J;
          const long n_end =
              sym ? (a.L >= band_len(J) ? min((a.L - band_len(J)) / (1L << J) + 1, nJf) : 0L) : nJf;
          band_tile<T, D, J>(Kunit, a.L, n0, ncoef, n_end, !sym, band, coef, map);
          // at most three edge coefficients: wave w takes the w-th of the tile
          const long n = max(n0, n_end) + (threadIdx.x >> 6);
          if (n < n0 + ncoef) edge_coef<T, D, J>(Kunit, n0, n, nJf, edge_lds, coef, map);
        } else {
          cascade_tile<M, J, T, D>(Kunit, a.L, n0, ncoef, a.cpt, sym, taps, coef, map);
        }
      };
      if (a.parent)
        transform(RowsGathered{a.parent + (long)u * a.npar, J + 1, a.Ls - 1});
      else
        transform(RowsIdentity{});
    } else {
      // the tile of A_J rows: every load issued before the first is waited
      // for (row indices clamped, stores guarded); with bf16 queries the
      // rows go straight to the [hi x D][lo x D] layout of split_tile_bf16
      const float* src = a.approx + ((long)u * a.nJ + n0) * D;
      constexpr int GPR = D / 8;  // 8-channel groups per row
      constexpr int MAXI = kMaxCoefTile * GPR / kBlock;
      f32x4 v0[MAXI], v1[MAXI];
#pragma unroll
      for (int k = 0; k < MAXI; ++k) {
        const int it = threadIdx.x + k * kBlock, row = min(it / GPR, ncoef - 1), grp = it % GPR;
        v0[k] = *reinterpret_cast<const f32x4*>(src + (long)row * D + 8 * grp);
        v1[k] = *reinterpret_cast<const f32x4*>(src + (long)row * D + 8 * grp + 4);
      }
#pragma unroll
      for (int k = 0; k < MAXI; ++k) {
        const int it = threadIdx.x + k * kBlock, row = it / GPR, grp = it % GPR;
        if (row >= ncoef) continue;
        if constexpr (sizeof(T) == 2) {
          const float v[8] = {v0[k][0], v0[k][1], v0[k][2], v0[k][3],
                              v1[k][0], v1[k][1], v1[k][2], v1[k][3]};
          uint32_t hi[4], lo[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            hi[e] = pack_bf16x2(v[2 * e], v[2 * e + 1]);
            lo[e] = pack_bf16x2(v[2 * e] - bf16_lo(hi[e]), v[2 * e + 1] - bf16_hi(hi[e]));
          }
          unsigned char* dst = reinterpret_cast<unsigned char*>(coef + row * (D + kCoefPad));
          *reinterpret_cast<u32x4*>(dst + 16 * grp) = u32x4{hi[0], hi[1], hi[2], hi[3]};
          *reinterpret_cast<u32x4*>(dst + 2 * D + 16 * grp) = u32x4{lo[0], lo[1], lo[2], lo[3]};
        } else {
          float* dst = coef + row * (D + kCoefPad) + 8 * grp;
          *reinterpret_cast<f32x4*>(dst) = v0[k];
          *reinterpret_cast<f32x4*>(dst + 4) = v1[k];
        }
      }
    }
    __syncthreads();
    if constexpr (sizeof(T) == 2 && SRC != kFromApprox) split_tile_bf16<D>(coef, ncoef);
    skim_epilogue<T, D>(a, u, tile, n0, ncoef, coef);
    __syncthreads();
  }
}

// Haar A_J alone (no details): block sums of 2^J rows in coefficient tiles
// (the same tiles the skim builds), then copied to approx [U][nJ][D].
// Persistent grid over (unit, tile) items.
template <typename T, int D>
__global__ __launch_bounds__(kBlock) void haar_approx_kernel(DwtArgs a, float inv_norm,
                                                             int cpt) {
  extern __shared__ float coef[];  // [cpt][D + kCoefPad]
  constexpr int STRIDE = D + kCoefPad;
  const int total = a.U * a.ntiles;
  for (int item = blockIdx.x; item < total; item += gridDim.x) {
    const int u = item / a.ntiles;
    const int tile = item % a.ntiles;
    const long n0 = (long)tile * cpt;
    const int ncoef = (int)min((long)cpt, (long)a.nJ - n0);
    const T* Kunit = reinterpret_cast<const T*>(a.K) + (long)u * a.Ls * D;
    haar_sum_tile<T, D>(Kunit, n0, ncoef, a.J, inv_norm, coef, [](long n) { return n; });
    __syncthreads();
    float* dst = a.approx + ((long)u * a.nJ + n0) * D;
    for (int v = threadIdx.x; v < ncoef * (D / 4); v += kBlock) {
      const int c = v / (D / 4), k = v % (D / 4);
      *reinterpret_cast<f32x4*>(dst + (long)c * D + 4 * k) =
          *reinterpret_cast<const f32x4*>(coef + c * STRIDE + 4 * k);
    }
    __syncthreads();
  }
}

// One workgroup per unit: merge the tiles' row statistics, form W (eq. 8) and
// select the top-S regions (eq. 9).
// W_j (eq. 8) of unit u for the columns 4 j4 .. 4 j4 + 3, j4 in [j4_lo,
// j4_hi) (nJ a multiple of 4), from the query-major logits and the row
// normalisers c_q = M_q log2(e) + log2(Z_q); also into wsh when given.
template <int NT>
__device__ void skim_w_columns(const SkimSelectArgs& a, int u, const float* row_c, int j4_lo,
                               int j4_hi, float* wsh) {
  const float* lg = a.logits + (long)u * a.B * a.nJ;
  float* W = a.W + (long)u * a.nJ;
  // four adjacent columns per thread, 16 query rows of loads in flight
  constexpr int QB = 16;
  for (int j4 = j4_lo + (int)threadIdx.x; j4 < j4_hi; j4 += NT) {
    float w[4] = {0.f, 0.f, 0.f, 0.f};
    for (int q0 = 0; q0 < a.B; q0 += QB) {
      float4 v[QB];
#pragma unroll
      for (int i = 0; i < QB; ++i)
        v[i] = q0 + i < a.B ? *reinterpret_cast<const float4*>(lg + (long)(q0 + i) * a.nJ + 4 * j4)
                            : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int i = 0; i < QB; ++i) {
        if (q0 + i < a.B) {
          const float c = row_c[q0 + i];
          w[0] += __builtin_amdgcn_exp2f(fmaf(v[i].x, kLog2e, -c));
          w[1] += __builtin_amdgcn_exp2f(fmaf(v[i].y, kLog2e, -c));
          w[2] += __builtin_amdgcn_exp2f(fmaf(v[i].z, kLog2e, -c));
          w[3] += __builtin_amdgcn_exp2f(fmaf(v[i].w, kLog2e, -c));
        }
      }
    }
    *reinterpret_cast<float4*>(W + 4 * j4) = make_float4(w[0], w[1], w[2], w[3]);
    if (wsh) {
#pragma unroll
      for (int e = 0; e < 4; ++e) wsh[4 * j4 + e] = w[e];
    }
  }
}

// Per query row of unit u: c_q = M_q log2(e) + log2(Z_q) of the coarse
// logits, from the tiles' (max, sum) slices, 64 rows at a time; thread
// (part, q) = (tid / 64, tid % 64) folds slices part, part + 4, ..., and the
// four parts meet in pm / pz.
__device__ void unit_row_norms(const SkimSelectArgs& a, int u, float* row_c, float (*pm)[64],
                               float (*pz)[64]) {
  const float* st = a.stats + (long)u * a.ntiles * 2 * a.B;
  for (int qc = 0; qc < a.B; qc += 64) {
    const int q = qc + (threadIdx.x & 63), pp = threadIdx.x >> 6;
    float m = -INFINITY, z = 0.f;
    if (q < a.B) {
      constexpr int BATCH = 8;
      for (int t0 = pp; t0 < a.ntiles; t0 += 4 * BATCH) {
        float tm[BATCH], tz[BATCH];
#pragma unroll
        for (int k = 0; k < BATCH; ++k) {
          const int t = t0 + 4 * k;
          tm[k] = t < a.ntiles ? st[(long)t * 2 * a.B + q] : -INFINITY;
          tz[k] = t < a.ntiles ? st[(long)t * 2 * a.B + a.B + q] : 0.f;
        }
#pragma unroll
        for (int k = 0; k < BATCH; ++k) pair_merge(m, z, tm[k], tz[k]);
      }
    }
    pm[pp][threadIdx.x & 63] = m;
    pz[pp][threadIdx.x & 63] = z;
    __syncthreads();
    if (threadIdx.x < 64 && q < a.B) {
      float mm = pm[0][threadIdx.x], zz = pz[0][threadIdx.x];
#pragma unroll
      for (int k = 1; k < 4; ++k) pair_merge(mm, zz, pm[k][threadIdx.x], pz[k][threadIdx.x]);
      row_c[q] = fmaf(mm, kLog2e, __log2f(zz));
    }
    __syncthreads();
  }
}

// W of a wide candidate set spread over `parts` workgroups per unit (the
// loads of one workgroup per unit would leave most CUs idle): every
// workgroup merges the unit's (max, sum) slices itself, then forms W for its
// share of the columns, four adjacent columns and every query row a thread.
__global__ __launch_bounds__(kBlock) void skim_weights_kernel(SkimSelectArgs a, int parts) {
  __shared__ float row_c[WF_MAX_Q_LEN];
  __shared__ float pm[4][64], pz[4][64];
  // a unit's parts on the XCD of the token skim that wrote its logits
  const int item = xcd_swizzle(blockIdx.x, gridDim.x);
  const int u = item / parts, part = item % parts;
  unit_row_norms(a, u, row_c, pm, pz);
  const int n4 = a.nJ / 4, per = (n4 + parts - 1) / parts;
  skim_w_columns<kBlock>(a, u, row_c, part * per, min(n4, (part + 1) * per), nullptr);
}

// The same W for a narrower candidate set (a thousand or so columns a unit),
// where a thread per four columns leaves too few threads: thread (g, c) adds
// the terms of query rows 16 g .. 16 g + 15 (and every 64th row after them)
// of four adjacent columns, the four groups' partial sums meet in LDS and are
// added in order of g.  The first batch of logits is loaded before the
// slices are merged, so that the two loads overlap.
__global__ __launch_bounds__(kBlock) void skim_weights_rows_kernel(SkimSelectArgs a, int parts) {
  constexpr int QB = 16;             // query rows of one batch
  constexpr int NQG = 4;             // query groups
  constexpr int CPW = kBlock / NQG;  // four-column groups per step
  __shared__ float row_c[WF_MAX_Q_LEN];
  __shared__ float pm[4][64], pz[4][64];
  __shared__ float4 wpart[NQG][CPW];
  const int item = xcd_swizzle(blockIdx.x, gridDim.x);
  const int u = item / parts, part = item % parts;
  const int n4 = a.nJ / 4, per = (n4 + parts - 1) / parts;
  const int j4_lo = part * per, j4_hi = min(n4, j4_lo + per);
  const int qg = threadIdx.x / CPW, cl = threadIdx.x % CPW;
  const float* lg = a.logits + (long)u * a.B * a.nJ;
  float4 v[QB];
  auto load = [&](int j4, int q0) {
#pragma unroll
    for (int i = 0; i < QB; ++i)
      v[i] = j4 < j4_hi && q0 + i < a.B
                 ? *reinterpret_cast<const float4*>(lg + (long)(q0 + i) * a.nJ + 4 * j4)
                 : make_float4(0.f, 0.f, 0.f, 0.f);
  };
  load(j4_lo + cl, QB * qg);
  unit_row_norms(a, u, row_c, pm, pz);

  float* W = a.W + (long)u * a.nJ;
  for (int s0 = j4_lo; s0 < j4_hi; s0 += CPW) {
    const int j4 = s0 + cl;
    float w[4] = {0.f, 0.f, 0.f, 0.f};
    for (int q0 = QB * qg; q0 < a.B; q0 += QB * NQG) {
      if (s0 != j4_lo || q0 != QB * qg) load(j4, q0);  // the first batch is in
#pragma unroll
      for (int i = 0; i < QB; ++i) {
        if (q0 + i < a.B) {
          // exp(l - M) / Z = 2^(l log2(e) - c)
          const float c = row_c[q0 + i];
          w[0] += __builtin_amdgcn_exp2f(fmaf(v[i].x, kLog2e, -c));
          w[1] += __builtin_amdgcn_exp2f(fmaf(v[i].y, kLog2e, -c));
          w[2] += __builtin_amdgcn_exp2f(fmaf(v[i].z, kLog2e, -c));
          w[3] += __builtin_amdgcn_exp2f(fmaf(v[i].w, kLog2e, -c));
        }
      }
    }
    wpart[qg][cl] = make_float4(w[0], w[1], w[2], w[3]);
    __syncthreads();
    if (qg == 0 && j4 < j4_hi) {
      float4 t = wpart[0][cl];
#pragma unroll
      for (int g = 1; g < NQG; ++g) {
        const float4 o = wpart[g][cl];
        t.x += o.x;
        t.y += o.y;
        t.z += o.z;
        t.w += o.w;
      }
      *reinterpret_cast<float4*>(W + 4 * j4) = t;
    }
    __syncthreads();
  }
}

constexpr int kSelectBlock = 1024;

__global__ __launch_bounds__(kSelectBlock) void skim_select_kernel(SkimSelectArgs a,
                                                                   int w_in_lds, int w_ready) {
  constexpr int NT = kSelectBlock;
  __shared__ float row_c[WF_MAX_Q_LEN];  // per query: M log2(e) + log2(Z)
  __shared__ float pm[16][65], pz[16][65];
  __shared__ SelectShared<NT> sh;
  extern __shared__ float wsh[];
  // the unit on the XCD whose L2 took its W (or its logits)
  const int u = xcd_swizzle(blockIdx.x, gridDim.x);
  const float* st = a.stats + (long)u * a.ntiles * 2 * a.B;
  float* W = a.W + (long)u * a.nJ;
  // candidate n is block n, or on a refinement scale child n % 2 of kept
  // block parent[n / 2]; the last scale emits the two tokens of each block
  int32_t* out = a.seg + (long)u * (a.pairs ? 2 : 1) * a.S;
  auto put = [&](uint32_t pos, int32_t id) {
    if (a.pairs) {
      out[2 * pos] = 2 * id;
      out[2 * pos + 1] = 2 * id + 1;
    } else {
      out[pos] = id;
    }
  };
  if (w_ready && a.nJ <= 8 * NT) {
    // W from skim_weights_kernel, eight scores a thread read once into
    // registers; the parent ids wait in LDS (the select's first barrier
    // orders them before any emit; n_J = 2 npar floats of LDS were sized)
    const int32_t* pg = a.parent ? a.parent + (long)u * a.npar : nullptr;
    int32_t* par_sh = reinterpret_cast<int32_t*>(wsh);
    if (pg)
      for (int i = threadIdx.x; i < a.npar; i += NT) par_sh[i] = pg[i];
    block_select_topk_regs<NT, 8>(
        W, a.nJ, a.S, [&](uint32_t pos, int n) { put(pos, pg ? 2 * par_sh[n >> 1] + (n & 1) : n); },
        sh);
    return;
  }
  if (w_ready) {
    // W was formed by skim_weights_kernel
    if (w_in_lds)
      for (int j = threadIdx.x; j < a.nJ; j += NT) wsh[j] = W[j];
  } else {
    // merge the tiles' (max, sum of exp) pairs, 64 queries at a time: thread
    // (part, q) = (tid / 64, tid % 64) folds tiles part, part + 16, ...; the 16
    // pairs of a query meet in a 16-lane row and are merged by rotations
    for (int qc = 0; qc < a.B; qc += 64) {
      {
        const int q = qc + (threadIdx.x & 63), part = threadIdx.x >> 6;
        float m = -INFINITY, z = 0.f;
        if (q < a.B) {
          constexpr int BATCH = 8;
          for (int t0 = part; t0 < a.ntiles; t0 += 16 * BATCH) {
            float tm[BATCH], tz[BATCH];
#pragma unroll
            for (int k = 0; k < BATCH; ++k) {
              const int t = t0 + 16 * k;
              tm[k] = t < a.ntiles ? st[(long)t * 2 * a.B + q] : -INFINITY;
              tz[k] = t < a.ntiles ? st[(long)t * 2 * a.B + a.B + q] : 0.f;
            }
#pragma unroll
            for (int k = 0; k < BATCH; ++k) pair_merge(m, z, tm[k], tz[k]);
          }
        }
        pm[part][threadIdx.x & 63] = m;
        pz[part][threadIdx.x & 63] = z;
      }
      __syncthreads();
      {
        const int ql = threadIdx.x >> 4, part = threadIdx.x & 15;
        float m = pm[part][ql], z = pz[part][ql];
        row16_merge<8>(m, z);
        row16_merge<4>(m, z);
        row16_merge<2>(m, z);
        row16_merge<1>(m, z);
        // exp(l - M) / Z = 2^(l log2(e) - c)
        if (part == 0 && qc + ql < a.B) row_c[qc + ql] = fmaf(m, kLog2e, __log2f(z));
      }
      __syncthreads();
    }
    const float* lg = a.logits + (long)u * a.B * a.nJ;
    if ((a.nJ & 3) == 0) {
      skim_w_columns<NT>(a, u, row_c, 0, a.nJ / 4, w_in_lds ? wsh : nullptr);
    } else {
      constexpr int RB = 16;  // rows in flight per thread
      for (int j = threadIdx.x; j < a.nJ; j += NT) {
        float w = 0.f;
        for (int q0 = 0; q0 < a.B; q0 += RB) {
          float v[RB];
#pragma unroll
          for (int i = 0; i < RB; ++i) v[i] = q0 + i < a.B ? lg[(long)(q0 + i) * a.nJ + j] : 0.f;
#pragma unroll
          for (int i = 0; i < RB; ++i)
            if (q0 + i < a.B) w += __builtin_amdgcn_exp2f(fmaf(v[i], kLog2e, -row_c[q0 + i]));
        }
        W[j] = w;
        if (w_in_lds) wsh[j] = w;
      }
    }
  }
  __syncthreads();
  const int32_t* par = a.parent ? a.parent + (long)u * a.npar : nullptr;
  auto emit = [&](uint32_t pos, int n) { put(pos, par ? 2 * par[n >> 1] + (n & 1) : n); };
  // one instance per address space of the weights
  if (w_in_lds)
    block_select_topk<kSelectBlock>(wsh, a.nJ, a.S, emit, sh);
  else
    block_select_topk<kSelectBlock>(W, a.nJ, a.S, emit, sh);
}

// ------------------------------------------------------------ host side

static Taps make_taps(int wavelet, int J) {
  Taps t{};
  const double r2 = std::sqrt(2.0);
  if (wavelet == WF_HAAR) {
    t.g[0] = t.g[1] = (float)(1.0 / r2);
    t.h[0] = (float)(1.0 / r2);
    t.h[1] = (float)(-1.0 / r2);
  } else {
    const double r3 = std::sqrt(3.0), den = 4.0 * r2;
    const double g[4] = {(1 + r3) / den, (3 + r3) / den, (3 - r3) / den,
                         (1 - r3) / den};
    for (int m = 0; m < 4; ++m) {
      t.g[m] = (float)g[m];
      t.h[m] = (float)((m % 2 == 0 ? 1.0 : -1.0) * g[3 - m]);
    }
  }
  t.inv_norm = (float)std::pow(2.0, -0.5 * J);
  return t;
}

// The three symmetric-end filters of the level-J Daubechies-2 approximation
// (see EdgeTaps), in double, once per J: impulses at each of the last 3 2^J
// rows of a sequence of 6 2^J rows, through the cascade with the
// half-sample symmetric extension at every level.
static const EdgeTaps& symmetric_edge_filters(int J) {
  static EdgeTaps table[kBandMaxJ + 1];
  static std::once_flag once[kBandMaxJ + 1];
  std::call_once(once[J], [J] {
    const double r2 = std::sqrt(2.0), r3 = std::sqrt(3.0), den = 4.0 * r2;
    const double g[4] = {(1 + r3) / den, (3 + r3) / den, (3 - r3) / den, (1 - r3) / den};
    const int blk = 1 << J, len = 6 * blk, nJ = 6;
    EdgeTaps& t = table[J];
    for (int i = 0; i < (6 << kBandMaxJ); ++i) t.e[i] = 0.f;
    for (int r = len - 3 * blk; r < len; ++r) {
      std::vector<double> y(len, 0.0);
      y[r] = 1.0;
      for (int j = 1; j <= J; ++j) {
        const int N = (int)y.size();
        std::vector<double> a(N / 2);
        for (int n = 0; n < N / 2; ++n) {
          double v = 0.0;
          for (int m = 0; m < 4; ++m) {
            const int i = 2 * n + m;
            v += g[m] * (i < N ? y[i] : y[2 * N - 1 - i]);
          }
          a[n] = v;
        }
        y.swap(a);
      }
      for (int m = 0; m < 3; ++m) {
        const int start = len - blk * (m + 1);  // first row of coefficient nJ - 1 - m
        if (r >= start) t.e[blk * (m * (m + 1) / 2) + (r - start)] = (float)y[nJ - 1 - m];
      }
    }
  });
  return table[J];
}

void db2_token_taps(int J, Db2TokenTaps* out) {
  const double r2 = std::sqrt(2.0), r3 = std::sqrt(3.0), den = 4.0 * r2;
  const double g[4] = {(1 + r3) / den, (3 + r3) / den, (3 - r3) / den, (1 - r3) / den};
  // f_1 = g, f_{j+1}[s] = sum_k g_k f_j[s - 2^j k]
  std::vector<double> f(g, g + 4);
  for (int j = 1; j < J; ++j) {
    std::vector<double> nf(f.size() + 3 * ((size_t)1 << j), 0.0);
    for (size_t s = 0; s < nf.size(); ++s)
      for (int k = 0; k < 4; ++k) {
        const long i = (long)s - ((long)k << j);
        if (i >= 0 && i < (long)f.size()) nf[s] += g[k] * f[i];
      }
    f.swap(nf);
  }
  for (int i = 0; i < (3 << 6); ++i) out->band[i] = i < (int)f.size() ? (float)f[i] : 0.f;
  const EdgeTaps& e = symmetric_edge_filters(J);
  for (int i = 0; i < (6 << 6); ++i) out->edge[i] = e.e[i];
}

template <int M, typename T>
static hipError_t dwt_dispatch(const DwtArgs& a, const Taps& taps, dim3 grid,
                               hipStream_t s) {
  switch (a.J) {
#define WF_DWT_CASE(JJ)                                                  \
  case JJ:                                                               \
    hipLaunchKernelGGL((dwt_kernel<M, JJ, T>), grid, dim3(kBlock), 0, s, \
                       a, taps);                                         \
    break;
    WF_DWT_CASE(1) WF_DWT_CASE(2) WF_DWT_CASE(3) WF_DWT_CASE(4)
    WF_DWT_CASE(5) WF_DWT_CASE(6) WF_DWT_CASE(7) WF_DWT_CASE(8)
    WF_DWT_CASE(9) WF_DWT_CASE(10)
#undef WF_DWT_CASE
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Haar coefficient tile size at level J.
static int haar_cpt(int J) { return std::min(kMaxCoefTile, std::max(16, 2048 >> J)); }
// coefficients per tile at scale b of the recursion
static int rec_cpt(const wf_params& p, int b) {
  return p.wavelet == WF_HAAR ? haar_cpt(b) : kMaxCoefTile;
}

DwtPlan plan_dwt(const wf_params& p) {
  DwtPlan d;
  const int spw = kWave / (p.head_dim / 2);
  d.streams = (kBlock / kWave) * spw;
  d.cps = std::max(1, 2048 >> p.levels);
  const long nJ = (long)p.ctx_len >> p.levels;
  const long per_tile = (long)d.streams * d.cps;
  d.ntiles = (int)((nJ + per_tile - 1) / per_tile);
  return d;
}

hipError_t launch_dwt(const wf_params& p, const void* K, float* approx,
                      float* details, hipStream_t s) {
  DwtPlan pl = plan_dwt(p);
  DwtArgs a;
  a.K = K;
  a.approx = approx;
  a.details = details;
  a.U = p.batch * p.heads;
  a.L = (int)filtered_len(p);
  a.Ls = p.ctx_len;
  a.D = p.head_dim;
  a.J = p.levels;
  a.nJ = p.ctx_len >> p.levels;
  a.cps = pl.cps;
  a.streams = pl.streams;
  a.ntiles = pl.ntiles;
  a.boundary = p.boundary;
  const Taps taps = make_taps(p.wavelet, p.levels);
  if (p.wavelet == WF_HAAR && !details) {
    // A_J is the scaled block sum: coefficient tiles at streaming rate
    const int cpt = haar_cpt(p.levels);
    a.ntiles = (int)((a.nJ + cpt - 1) / cpt);
    const size_t lds = (size_t)cpt * (p.head_dim + kCoefPad) * sizeof(float);
    auto run = [&](auto kern) -> hipError_t {
      int per_cu = 0;
      hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &per_cu, reinterpret_cast<const void*>(kern), kBlock, lds);
      if (e != hipSuccess) return e;
      const long total = (long)a.U * a.ntiles;
      const long cap = (long)std::max(1, per_cu) * device_cu_count();
      hipLaunchKernelGGL(kern, dim3((unsigned)std::min(total, cap)), dim3(kBlock), lds, s, a,
                         taps.inv_norm, cpt);
      return hipGetLastError();
    };
    if (p.dtype == WF_BF16)
      return p.head_dim == 128 ? run(haar_approx_kernel<bf16_t, 128>)
                               : run(haar_approx_kernel<bf16_t, 64>);
    return p.head_dim == 128 ? run(haar_approx_kernel<float, 128>)
                             : run(haar_approx_kernel<float, 64>);
  }
  dim3 grid((unsigned)(a.U * a.ntiles));
  const bool haar = p.wavelet == WF_HAAR;
  if (p.dtype == WF_BF16)
    return haar ? dwt_dispatch<2, bf16_t>(a, taps, grid, s)
                : dwt_dispatch<4, bf16_t>(a, taps, grid, s);
  return haar ? dwt_dispatch<2, float>(a, taps, grid, s)
              : dwt_dispatch<4, float>(a, taps, grid, s);
}

SkimPlan plan_skim(const wf_params& p, bool fused) {
  SkimPlan k;
  const int J = p.levels;
  if (!fused) {
    k.source = kFromApprox;
    k.cpt = kMaxCoefTile;
  } else if (p.wavelet == WF_HAAR) {
    k.source = kHaarSum;
    k.cpt = std::min(kMaxCoefTile, std::max(16, 2048 >> J));
  } else {
    k.source = kCascade;
    k.cpt = kMaxCoefTile;  // 4 (d=128) or 8 (d=64) streams of 16 or 8
  }
  const long nJ = (long)p.ctx_len >> J;
  k.ntiles = (int)((nJ + k.cpt - 1) / k.cpt);
  k.lds_bytes = ((size_t)k.cpt * (p.head_dim + kCoefPad) +
                 (k.source == kCascade ? (size_t)12 << J : 0)) * sizeof(float);
  return k;
}

template <int SRC, int M, int J, typename T, int D>
static hipError_t skim_launch_one(const SkimTileArgs& a, const Taps& taps, const EdgeTaps& edge,
                                  size_t lds, hipStream_t s) {
  auto kern = skim_tile_kernel<SRC, M, J, T, D>;
  int per_cu = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
      &per_cu, reinterpret_cast<const void*>(kern), kBlock, lds);
  if (e != hipSuccess) return e;
  const long total = (long)a.U * a.ntiles;
  const long cap = (long)std::max(1, per_cu) * device_cu_count();
  dim3 grid((unsigned)std::min(total, cap));
  hipLaunchKernelGGL(kern, grid, dim3(kBlock), lds, s, a, taps, edge);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t skim_dispatch(int source, const SkimTileArgs& a, const Taps& taps,
                                const EdgeTaps& edge, size_t lds, hipStream_t s) {
  if (source == kHaarSum) return skim_launch_one<kHaarSum, 2, 1, T, D>(a, taps, edge, lds, s);
  if (source == kFromApprox)
    return skim_launch_one<kFromApprox, 2, 1, T, D>(a, taps, edge, lds, s);
  switch (a.J) {
#define WF_SKIM_CASE(JJ) \
  case JJ:               \
    return skim_launch_one<kCascade, 4, JJ, T, D>(a, taps, edge, lds, s);
    WF_SKIM_CASE(1) WF_SKIM_CASE(2) WF_SKIM_CASE(3) WF_SKIM_CASE(4)
    WF_SKIM_CASE(5) WF_SKIM_CASE(6) WF_SKIM_CASE(7) WF_SKIM_CASE(8)
    WF_SKIM_CASE(9) WF_SKIM_CASE(10)
#undef WF_SKIM_CASE
    default:
      return hipErrorInvalidValue;
  }
}

static hipError_t skim_tiles_common(const wf_params& p, int source, int cpt, int J,
                                    long nJ, const int32_t* parent, int npar,
                                    const void* Q, const void* K, const float* approx,
                                    float* logits, float* stats, hipStream_t s) {
  SkimTileArgs a;
  a.K = K;
  a.approx = approx;
  a.Q = Q;
  a.logits = logits;
  a.stats = stats;
  a.parent = parent;
  a.npar = npar;
  a.U = p.batch * p.heads;
  // rows transformed: the filtered keys, or for the db2 filter on a
  // refinement scale of the recursion the gathered kept blocks of 2^(J+1)
  // rows each (Haar sums read the kept blocks' halves in place)
  a.L = parent && source == kCascade ? (int)((long)npar << (J + 1)) : (int)filtered_len(p);
  a.Ls = p.ctx_len;
  a.B = p.q_len;
  a.J = J;
  a.nJ = (int)nJ;
  a.cpt = cpt;
  a.ntiles = (int)((nJ + cpt - 1) / cpt);
  a.boundary = p.boundary;
  a.scale = effective_scale(p);
  // the coefficient tile, then (cascade source) the banded filter's taps
  // and the symmetric-end filters
  const size_t lds = ((size_t)cpt * (p.head_dim + kCoefPad) +
                      (source == kCascade ? (size_t)12 << J : 0)) *
                     sizeof(float);
  const Taps taps = make_taps(p.wavelet, J);
  static const EdgeTaps no_edge{};
  const EdgeTaps& edge = source == kCascade && p.wavelet == WF_DB2 &&
                                 p.boundary == WF_EXT_SYMMETRIC && J <= kBandMaxJ
                             ? symmetric_edge_filters(J)
                             : no_edge;
  if (p.dtype == WF_BF16)
    return p.head_dim == 128 ? skim_dispatch<bf16_t, 128>(source, a, taps, edge, lds, s)
                             : skim_dispatch<bf16_t, 64>(source, a, taps, edge, lds, s);
  return p.head_dim == 128 ? skim_dispatch<float, 128>(source, a, taps, edge, lds, s)
                           : skim_dispatch<float, 64>(source, a, taps, edge, lds, s);
}

hipError_t launch_skim_tiles(const wf_params& p, bool fused, const void* Q,
                             const void* K, const float* approx, float* logits,
                             float* stats, hipStream_t s) {
  const SkimPlan pl = plan_skim(p, fused);
  return skim_tiles_common(p, pl.source, pl.cpt, p.levels, (long)p.ctx_len >> p.levels,
                           nullptr, 0, Q, K, approx, logits, stats, s);
}

static hipError_t skim_select_common(const wf_params& p, long nJ, int ntiles, int S,
                                     const int32_t* parent, int npar, int pairs,
                                     const float* logits, const float* stats, float* W,
                                     int32_t* out, hipStream_t s) {
  SkimSelectArgs a;
  a.logits = logits;
  a.stats = stats;
  a.W = W;
  a.seg = out;
  a.parent = parent;
  a.npar = npar;
  a.pairs = pairs;
  a.U = p.batch * p.heads;
  a.B = p.q_len;
  a.nJ = (int)nJ;
  a.ntiles = ntiles;
  a.S = S;
  const int in_lds = a.nJ <= kSelectLdsFloats ? 1 : 0;
  const size_t lds = in_lds ? (size_t)a.nJ * sizeof(float) : 0;
  if (lds > 32768) {  // with the static arrays, past the default 64 KiB
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(skim_select_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  // wide candidate sets: W over all CUs first (1024 columns a workgroup)
  const int w_ready = a.nJ >= 4096 && (a.nJ & 3) == 0 ? 1 : 0;
  if (w_ready) {
    const int parts = (a.nJ + 1023) / 1024;
    hipLaunchKernelGGL(skim_weights_kernel, dim3((unsigned)(a.U * parts)), dim3(kBlock), 0, s,
                       a, parts);
  }
  hipLaunchKernelGGL(skim_select_kernel, dim3((unsigned)a.U), dim3(kSelectBlock),
                     lds, s, a, in_lds, w_ready);
  return hipGetLastError();
}

hipError_t launch_select_w(const wf_params& p, long groups, const float* W, int32_t* seg,
                           hipStream_t s) {
  if (groups < 1 || !W || !seg) return hipErrorInvalidValue;
  SkimSelectArgs a{};
  a.W = const_cast<float*>(W);
  a.seg = seg;
  a.U = (int)groups;
  a.B = p.q_len;
  a.nJ = (int)((long)p.ctx_len >> p.levels);
  a.S = p.segments;
  const int in_lds = a.nJ <= kSelectLdsFloats ? 1 : 0;
  const size_t lds = in_lds ? (size_t)a.nJ * sizeof(float) : 0;
  if (lds > 32768) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(skim_select_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(skim_select_kernel, dim3((unsigned)a.U), dim3(kSelectBlock), lds, s, a,
                     in_lds, 1);
  return hipGetLastError();
}

hipError_t launch_skim_weights(const wf_params& p, int ntiles, const float* logits,
                               const float* stats, float* W, hipStream_t s) {
  SkimSelectArgs a{};
  a.logits = logits;
  a.stats = stats;
  a.W = W;
  a.U = p.batch * p.heads;
  a.B = p.q_len;
  a.nJ = (int)((long)p.ctx_len >> p.levels);
  a.ntiles = ntiles;
  if (!logits || !stats || !W || (a.nJ & 3) != 0 || a.nJ == 0) return hipErrorInvalidValue;
  // at most 1024 columns a workgroup, and two workgroups per CU at least
  const long n4 = a.nJ / 4;
  const long want = std::max((a.nJ + 1023L) / 1024,
                             (2L * device_cu_count() + a.U - 1) / a.U);
  const int parts = (int)std::min(n4, want);
  hipLaunchKernelGGL(skim_weights_rows_kernel, dim3((unsigned)(a.U * parts)), dim3(kBlock), 0,
                     s, a, parts);
  return hipGetLastError();
}

hipError_t launch_skim_select(const wf_params& p, int ntiles,
                              const float* logits, const float* stats,
                              float* W, int32_t* seg, hipStream_t s) {
  return skim_select_common(p, (long)p.ctx_len >> p.levels, ntiles, p.segments, nullptr, 0,
                            0, logits, stats, W, seg, s);
}

RecPlan plan_recursion(const wf_params& p, const int32_t* counts) {
  RecPlan r{};
  long n = (long)p.ctx_len >> p.levels;
  for (int b = p.levels; b >= 1; --b) {
    const int cpt = rec_cpt(p, b);
    // with token logits the statistics come from the token skim's ranges
    const int ntiles =
        rec_token_path(p) && b <= 5
            ? plan_rec_token(p, b, b == p.levels ? filtered_len(p) : n << b, b != p.levels).R
            : (int)((n + cpt - 1) / cpt);
    r.max_n = std::max(r.max_n, n);
    r.max_tiles = std::max(r.max_tiles, ntiles);
    r.max_keep = std::max(r.max_keep, (long)counts[b - 1]);
    n = 2L * counts[b - 1];
  }
  return r;
}

hipError_t launch_rec_tiles(const wf_params& p, int b, long n, const int32_t* parent,
                            int npar, const void* Q, const void* K, float* logits,
                            float* stats, hipStream_t s) {
  return skim_tiles_common(p, p.wavelet == WF_HAAR ? kHaarSum : kCascade, rec_cpt(p, b), b, n,
                           parent, npar, Q, K, nullptr, logits, stats, s);
}

hipError_t launch_rec_select(const wf_params& p, int b, long n, int keep,
                             const int32_t* parent, int npar, const float* logits,
                             const float* stats, float* W, int32_t* out, hipStream_t s) {
  const int cpt = rec_cpt(p, b);
  const int ntiles = (int)((n + cpt - 1) / cpt);
  return skim_select_common(p, n, ntiles, keep, parent, npar, b == 1 ? 1 : 0, logits,
                            stats, W, out, s);
}
hipError_t launch_rec_select_slices(const wf_params& p, int b, long n, int keep,
                                    const int32_t* parent, int npar, int nslices,
                                    const float* logits, const float* stats, float* W,
                                    int32_t* out, hipStream_t s) {
  return skim_select_common(p, n, nslices, keep, parent, npar, b == 1 ? 1 : 0, logits,
                            stats, W, out, s);
}

hipError_t load_skim_kernels() {
  hipFuncAttributes fa;
  return hipFuncGetAttributes(&fa, reinterpret_cast<const void*>(skim_select_kernel));
}

}  // namespace wf
