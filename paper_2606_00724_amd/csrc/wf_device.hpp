// Device building blocks shared by the WaveFilter gfx950 kernels: element
// conversions, 16x16 MFMA tile products, a block-wide scan and a
// deterministic top-k selection.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wf {

constexpr int kWave = 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

struct bf16_t {
  uint16_t bits;
};

// ------------------------------------------------------------ conversions

__device__ __forceinline__ float bf16_lo(uint32_t w) {
  return __uint_as_float(w << 16);
}
__device__ __forceinline__ float bf16_hi(uint32_t w) {
  return __uint_as_float(w & 0xffff0000u);
}

// Round-to-nearest-even float -> bf16 bits (NaN stays NaN).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// Two floats to packed bf16 with one v_cvt_pk_bf16_f32: round to nearest
// even, bit-identical to f32_to_bf16_bits for every finite input (NaNs stay
// NaNs, possibly with another payload).
typedef __bf16 hw_bf16x2 __attribute__((ext_vector_type(2)));
typedef float hw_f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((hw_f32x2{lo, hi}), hw_bf16x2));
}

template <typename T>
__device__ __forceinline__ float load_elem(const T* p, long i);
template <>
__device__ __forceinline__ float load_elem<float>(const float* p, long i) {
  return p[i];
}
template <>
__device__ __forceinline__ float load_elem<bf16_t>(const bf16_t* p, long i) {
  return __uint_as_float((uint32_t)p[i].bits << 16);
}

template <typename T>
__device__ __forceinline__ void store_elem(T* p, long i, float v);
template <>
__device__ __forceinline__ void store_elem<float>(float* p, long i, float v) {
  p[i] = v;
}
template <>
__device__ __forceinline__ void store_elem<bf16_t>(bf16_t* p, long i, float v) {
  p[i].bits = (uint16_t)f32_to_bf16_bits(v);
}

// ------------------------------------------------------------ MFMA tiles
//
// A 16x16 output tile C[m][n] = sum_c Arow_m[c] * Brow_n[c], where lane l
// supplies row m = l % 16 of A and row n = l % 16 of B (both stored with
// channels contiguous).  On return lane l holds C[4 (l / 16) + i][l % 16] in
// element i.
//
// bf16 rows use v_mfma_f32_16x16x32_bf16: lane group g = l / 16 feeds
// channels 8g .. 8g+7 of every 32-channel step.  fp32 rows use
// v_mfma_f32_16x16x4_f32 with the channel order permuted so that lane group g
// walks the contiguous channel range [g D/4, (g+1) D/4): the reduction runs
// over every channel exactly once either way.

template <int D>
__device__ __forceinline__ f32x4 tile_dot_bf16(const bf16_t* a_row,
                                               const bf16_t* b_row,
                                               f32x4 acc) {
  const int g = (threadIdx.x & 63) >> 4;
#pragma unroll
  for (int s = 0; s < D / 32; ++s) {
    u32x4 a = *reinterpret_cast<const u32x4*>(a_row + 32 * s + 8 * g);
    u32x4 b = *reinterpret_cast<const u32x4*>(b_row + 32 * s + 8 * g);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
        __builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), acc, 0,
        0, 0);
  }
  return acc;
}

template <int D>
__device__ __forceinline__ f32x4 tile_dot_f32(const float* a_row,
                                              const float* b_row, f32x4 acc) {
  const int g = (threadIdx.x & 63) >> 4;
  const float* a = a_row + g * (D / 4);
  const float* b = b_row + g * (D / 4);
#pragma unroll
  for (int s4 = 0; s4 < D / 16; ++s4) {
    f32x4 av = *reinterpret_cast<const f32x4*>(a + 4 * s4);
    f32x4 bv = *reinterpret_cast<const f32x4*>(b + 4 * s4);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[e], bv[e], acc, 0, 0, 0);
  }
  return acc;
}

template <typename T, int D>
__device__ __forceinline__ f32x4 tile_dot(const T* a_row, const T* b_row,
                                          f32x4 acc);
template <>
__device__ __forceinline__ f32x4 tile_dot<bf16_t, 64>(const bf16_t* a,
                                                      const bf16_t* b,
                                                      f32x4 c) {
  return tile_dot_bf16<64>(a, b, c);
}
template <>
__device__ __forceinline__ f32x4 tile_dot<bf16_t, 128>(const bf16_t* a,
                                                       const bf16_t* b,
                                                       f32x4 c) {
  return tile_dot_bf16<128>(a, b, c);
}
template <>
__device__ __forceinline__ f32x4 tile_dot<float, 64>(const float* a,
                                                     const float* b, f32x4 c) {
  return tile_dot_f32<64>(a, b, c);
}
template <>
__device__ __forceinline__ f32x4 tile_dot<float, 128>(const float* a,
                                                      const float* b,
                                                      f32x4 c) {
  return tile_dot_f32<128>(a, b, c);
}

constexpr float kLog2e = 1.44269504088896341f;  // log2(e)
constexpr float kLn2 = 0.69314718055994531f;     // ln(2)

// one running (max, sum of exp) pair absorbs another
__device__ __forceinline__ void stat_absorb(float& m, float& z, float m2, float z2) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;
  z = (m > -INFINITY ? z * __expf(m - mn) : 0.f) + (m2 > -INFINITY ? z2 * __expf(m2 - mn) : 0.f);
  m = mn;
}

// ------------------------------------------------------------ reductions

// The value of the lane R lanes away (mod 16) in the same 16-lane row (DPP
// row_ror:R).
template <int R>
__device__ __forceinline__ float dpp_row_ror(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x120 + R, 0xf, 0xf, false));
}

// Max / sum over the 16 lanes of the lane's row, on DPP rotations (every
// lane ends with the row's result; every lane of the wave must be active).
// The sum's association order differs between the lanes of a row.
__device__ __forceinline__ float wave_max16(float v) {
  v = fmaxf(v, dpp_row_ror<8>(v));
  v = fmaxf(v, dpp_row_ror<4>(v));
  v = fmaxf(v, dpp_row_ror<2>(v));
  return fmaxf(v, dpp_row_ror<1>(v));
}
__device__ __forceinline__ float wave_sum16(float v) {
  v += dpp_row_ror<8>(v);
  v += dpp_row_ror<4>(v);
  v += dpp_row_ror<2>(v);
  return v + dpp_row_ror<1>(v);
}

// W (eq. 8) of blocks j0 .. j1 - 1 of one unit from the token skim's block
// rows lg [nJ][2][B] (coarse logits at 2 j B) and the unit's R range pairs
// ws [R][2][B] of (max, sum of exp) of its coarse logits per query:
// W_j = sum_q exp(l_qj - M_q) / Z_q, with (M_q, Z_q) the ranges' pairs
// merged.  A 16-lane row per block j, lane i holding queries 4 i .. 4 i + 3,
// so that a wave's loads cover whole block rows; the lanes' sums meet by DPP
// rotations (2^-inf = 0 for queries past B <= 64).  row_c: B floats of LDS.
// Every thread of the NT-thread block calls it (it has barriers); out(j, w)
// is called by one lane per block.
template <int NT, typename Out>
__device__ __forceinline__ void unit_block_weights(const float* lg, const float* ws, int R, int B,
                                                   int j0, int j1, float* row_c, Out out) {
  const int l16 = threadIdx.x & 15, grp = threadIdx.x >> 4;
  constexpr int G16 = NT / 16;  // blocks per round
  constexpr int RPT = 8;        // rounds whose loads are in flight together
  const bool vec = (B & 3) == 0;  // rows are 16-byte aligned
  float4 x[RPT];
  auto load = [&](int jb) {
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
      const int j = jb + r * G16 + grp;
      const float* row = lg + (long)j * 2 * B + 4 * l16;
      if (j < j1 && 4 * l16 < B) {
        if (vec) {
          x[r] = *reinterpret_cast<const float4*>(row);
        } else {
          x[r].x = row[0];
          x[r].y = 4 * l16 + 1 < B ? row[1] : -INFINITY;
          x[r].z = 4 * l16 + 2 < B ? row[2] : -INFINITY;
          x[r].w = 4 * l16 + 3 < B ? row[3] : -INFINITY;
        }
      } else {
        x[r] = float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      }
    }
  };
  // the first rounds load while the normalisers are merged
  load(j0);
  if (threadIdx.x < B) {
    // the ranges' pairs of query q, loads in flight together
    const int q = threadIdx.x;
    float mx = -INFINITY, z = 0.f;
    constexpr int SB = 8;
    for (int r0 = 0; r0 < R; r0 += SB) {
      float mr[SB], zr[SB];
#pragma unroll
      for (int k = 0; k < SB; ++k) {
        const bool ok = r0 + k < R;
        mr[k] = ok ? ws[(long)(r0 + k) * 2 * B + q] : -INFINITY;
        zr[k] = ok ? ws[(long)(r0 + k) * 2 * B + B + q] : 0.f;
      }
#pragma unroll
      for (int k = 0; k < SB; ++k) stat_absorb(mx, z, mr[k], zr[k]);
    }
    // exp(l - M_q) / Z_q = 2^(l log2(e) - c_q)
    row_c[q] = fmaf(mx, kLog2e, __log2f(z));
  }
  __syncthreads();
  float cq[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) cq[e] = 4 * l16 + e < B ? row_c[4 * l16 + e] : INFINITY;
  for (int jb = j0; jb < j1; jb += RPT * G16) {
    if (jb != j0) load(jb);
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
      const int j = jb + r * G16 + grp;
      float w = __builtin_amdgcn_exp2f(fmaf(x[r].x, kLog2e, -cq[0])) +
                __builtin_amdgcn_exp2f(fmaf(x[r].y, kLog2e, -cq[1])) +
                __builtin_amdgcn_exp2f(fmaf(x[r].z, kLog2e, -cq[2])) +
                __builtin_amdgcn_exp2f(fmaf(x[r].w, kLog2e, -cq[3]));
      w = wave_sum16(w);
      if (l16 == 0 && j < j1) out(j, w);
    }
  }
}

// Sums of v over lane pairs (l, l ^ 1) and (l, l ^ 2), DPP quad_perm.
__device__ __forceinline__ float add_xor1(float v) {
  return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xf, 0xf, false));
}
__device__ __forceinline__ float add_xor2(float v) {
  return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xf, 0xf, false));
}

// Reductions over the lane pairs (l, l ^ 16) and (l, l ^ 32) on the VALU:
// v_permlane16_swap / v_permlane32_swap of a value with itself leave the
// two partners' values in the two results (lane l gets {v[l], v[l ^ 16]} and
// {v[l % 32], v[l % 32 + 32]}), so no LDS round trip is needed. Every lane of
// the wave must be active.
__device__ __forceinline__ float max_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float add_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float add_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// The value of lane l ^ 32.
__device__ __forceinline__ float partner32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float((threadIdx.x & 32) ? r[0] : r[1]);
}

// Merges the (max, sum of exp) pair (m2, z2) into (m, z); empty pairs have
// m = -inf.
__device__ __forceinline__ void pair_merge(float& m, float& z, float m2, float z2) {
  const float mn = fmaxf(m, m2);
  if (mn > -INFINITY) {
    z = (m > -INFINITY ? z * __expf(m - mn) : 0.f) + (m2 > -INFINITY ? z2 * __expf(m2 - mn) : 0.f);
    m = mn;
  }
}

// Merges into the lane's (max, sum of exp) pair the pair R lanes away (mod 16) in its
// 16-lane row (DPP row_ror:R; every lane must be active).
template <int R>
__device__ __forceinline__ void row16_merge(float& m, float& z) {
  const float m2 = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(m), 0x120 + R, 0xf, 0xf, false));
  const float z2 = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(z), 0x120 + R, 0xf, 0xf, false));
  pair_merge(m, z, m2, z2);
}

// Order-preserving map of a float to uint32 (larger float -> larger key).
__device__ __forceinline__ uint32_t order_key(float x) {
  uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

template <int NT>
struct SelectShared {
  uint32_t hist[3][256];          // digit histograms, used in turn by the passes
  uint32_t cnt[2][8 * (NT / 64)]; // per-(round, wave) packed counts, used in turn by tiles
};

// Inclusive prefix sum over the 64 lanes of a wave, on DPP (no LDS round
// trips): shifts by 1, 2, 4, 8 inside each 16-lane row, then row 0's total
// into row 1 and row 2's into row 3 (row_bcast:15), then the first two
// rows' total into rows 2 and 3 (row_bcast:31).  Every lane must be active.
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, false);  // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return x;
}

// c[j] for a lane-varying j < 4, without indexing a register array
__device__ __forceinline__ uint32_t pick4(const uint32_t (&c)[4], int j) {
  return j == 0 ? c[0] : j == 1 ? c[1] : j == 2 ? c[2] : c[3];
}

// One count into bin d of the LDS histogram h for every active lane with m
// set.  When at least 8 of the wave's counting lanes share the digit of its
// first counting lane, they add as one atomic carrying the group's size and
// the rest add one each; otherwise every lane adds one.  Clustered keys
// (equal or nearly equal scores) would otherwise queue most of a wave's
// atomics on one LDS address.
__device__ __forceinline__ void hist_add(uint32_t* h, bool m, uint32_t d, int lane) {
  const uint64_t act = __builtin_amdgcn_ballot_w64(m);
  if (act == 0) return;  // uniform
  const int lead = __ffsll((unsigned long long)act) - 1;
  const uint32_t ld = (uint32_t)__builtin_amdgcn_readlane((int)d, lead);
  const bool mine = m && d == ld;
  const uint32_t group = (uint32_t)__popcll(__builtin_amdgcn_ballot_w64(mine));
  if (group >= 8) {  // uniform
    if (lane == lead) atomicAdd(&h[ld], group);
    if (m && !mine) atomicAdd(&h[d], 1u);
  } else if (m) {
    atomicAdd(&h[d], 1u);
  }
}

// Picks the k largest of score[0..n) (ties: lower index first) and calls
// emit(pos, i) for each picked position i, pos = its rank in ascending order
// of i (0..k-1).  Requires 1 <= k <= n and 64 <= NT <= 1024.  score may live in LDS or
// global memory; it must be visible to the whole block, and every thread of
// the block must call this.
//
// Radix select on order-preserving keys, one 8-bit digit per pass from the
// top: the candidates' digit histogram is built with LDS atomics, then every
// wave scans the 256 bins itself to find the digit holding the need-th
// largest candidate, so a pass costs one barrier (three histograms rotate so
// that the next one is cleared while the current one fills).  The last pass
// leaves the k-th largest key and the number of its copies to take; the
// passes stop early once the bin they narrowed to is taken whole (its keys'
// lower digits then change nothing, and keys compare under the digits
// resolved so far).  The output positions then follow from a scan of packed
// (greater, equal) counts over the positions in index order:
//   pos = #greater before + min(#equal before, copies to take).
template <int NT, typename Emit>
__device__ __forceinline__ void block_select_topk(const float* score, int n, int k, Emit emit,
                                  SelectShared<NT>& sh) {
  static_assert(NT >= 64 && NT <= 1024 && NT % 64 == 0, "block of whole waves");
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  for (int i = tid; i < 256; i += NT) sh.hist[0][i] = 0;
  __syncthreads();
  uint32_t prefix = 0, mask = 0, need = (uint32_t)k;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    uint32_t* h = sh.hist[pass % 3];
    // the histogram of the next pass was last read two passes ago
    if (pass < 3)
      for (int i = tid; i < 256; i += NT) sh.hist[(pass + 1) % 3][i] = 0;
    // batches of eight elements per thread whose loads are issued together
    // (a load under a per-lane condition would be waited for at once): lanes
    // past n load the last score and count nothing
    for (int b0 = 0; b0 < n; b0 += 8 * NT) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (b0 + u * NT < n) v[u] = score[min(b0 + u * NT + tid, n - 1)];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (b0 + u * NT >= n) break;  // uniform
        const uint32_t key = order_key(v[u]);
        hist_add(h, b0 + u * NT + tid < n && (key & mask) == prefix, (key >> shift) & 255u,
                 lane);
      }
    }
    __syncthreads();
    // lane l looks at digits 255 - 4l - j, j < 4 (descending)
    uint32_t c[4], sum = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      c[j] = h[255 - 4 * lane - j];
      sum += c[j];
    }
    uint32_t before = wave_inclusive_scan(sum) - sum;
    int hit = 0;
    uint32_t hit_above = 0;
    bool found = false;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (!found && before < need && before + c[j] >= need) {
        found = true;
        hit = j;
        hit_above = before;
      }
      before += c[j];
    }
    const int src = __ffsll((unsigned long long)__ballot(found)) - 1;
    // src is uniform: read the lane's values without an LDS round trip
    const uint32_t digit = (uint32_t)__builtin_amdgcn_readlane(255 - 4 * lane - hit, src);
    const uint32_t above = (uint32_t)__builtin_amdgcn_readlane((int)hit_above, src);
    const uint32_t in_bin = (uint32_t)__builtin_amdgcn_readlane((int)pick4(c, hit), src);
    prefix |= digit << shift;
    mask |= 255u << shift;
    need -= above;
    // every key of the bin is taken: its lower digits decide nothing
    if (need == in_bin) break;  // uniform
  }
  // the top keys are those above prefix under mask, and `need` of those
  // equal to it under mask (all of them when the passes stopped early).
  // Ordered compaction in tiles of ROUNDS x NT positions: position
  // base + j NT + tid is round j of the thread.  Each wave ballots its
  // (greater, equal) flags per round; one scan over the packed per-(round,
  // wave) counts, in index order, gives every wave its offsets, and a lane's
  // place inside its wave is the popcount of the ballot below it.
  constexpr int NW = NT / 64;
  constexpr int ROUNDS = 8;              // per-tile counts stay below 2^16
  constexpr int NE = ROUNDS * NW;        // entries of the count scan (<= 128)
  static_assert(NE <= 256, "count scan: at most four entries per lane");
  uint32_t gt_base = 0, eq_base = 0;
  int tile = 0;
  for (int base = 0; base < n; base += ROUNDS * NT, ++tile) {
    uint64_t gtm[ROUNDS], eqm[ROUNDS];
    uint32_t mine = 0;  // lane j < ROUNDS: the wave's packed counts of round j
    float v[ROUNDS];
#pragma unroll
    for (int j = 0; j < ROUNDS; ++j)
      if (base + j * NT < n) v[j] = score[min(base + j * NT + tid, n - 1)];
#pragma unroll
    for (int j = 0; j < ROUNDS; ++j) {
      const int i = base + j * NT + tid;
      bool gt = false, eq = false;
      if (base + j * NT < n && i < n) {
        const uint32_t key = order_key(v[j]) & mask;
        gt = key > prefix;
        eq = key == prefix;
      }
      gtm[j] = __ballot(gt);
      eqm[j] = __ballot(eq);
      if (lane == j) mine = ((uint32_t)__popcll(gtm[j]) << 16) | (uint32_t)__popcll(eqm[j]);
    }
    uint32_t* cnt = sh.cnt[tile & 1];  // [ROUNDS][NW]
    if (lane < ROUNDS) cnt[lane * NW + wid] = mine;
    __syncthreads();
    // exclusive scan of the NE entries (entry e = j NW + w), four per lane
    uint32_t c[4], sum = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * lane + q;
      c[q] = e < NE ? cnt[e] : 0u;
      sum += c[q];
    }
    const uint32_t incl = wave_inclusive_scan(sum);
    const uint32_t total = (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
    uint32_t ex[4];
    ex[0] = incl - sum;
#pragma unroll
    for (int q = 1; q < 4; ++q) ex[q] = ex[q - 1] + c[q - 1];
#pragma unroll
    for (int j = 0; j < ROUNDS; ++j) {
      if (base + j * NT >= n) break;  // uniform
      const int e = j * NW + wid;   // uniform
      const int q = e & 3;
      const uint32_t pick = q == 0 ? ex[0] : q == 1 ? ex[1] : q == 2 ? ex[2] : ex[3];
      const uint32_t off = (uint32_t)__builtin_amdgcn_readlane((int)pick, e >> 2);
      const uint64_t gm = gtm[j], em = eqm[j];
      const bool gt = (gm >> lane) & 1ull, eq = (em >> lane) & 1ull;
      const uint32_t gt_before = gt_base + (off >> 16) +
          __builtin_amdgcn_mbcnt_hi((uint32_t)(gm >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)gm, 0u));
      const uint32_t eq_before = eq_base + (off & 0xffffu) +
          __builtin_amdgcn_mbcnt_hi((uint32_t)(em >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)em, 0u));
      if (gt || (eq && eq_before < need)) {
        const uint32_t pos = gt_before + min(eq_before, need);
        if (pos < (uint32_t)k) emit(pos, base + j * NT + tid);
      }
    }
    gt_base += total >> 16;
    eq_base += total & 0xffffu;
  }
}

// block_select_topk for n <= EPT * NT with every key held in registers:
// element j NT + tid is slot j of thread tid, read once (from LDS or global
// memory), and every loop over the elements is unrolled.  Same picks, same
// emit positions (the same radix passes and ordered compaction).
template <int NT, int EPT, typename Emit>
__device__ __forceinline__ void block_select_topk_regs(const float* score, int n, int k, Emit emit,
                                       SelectShared<NT>& sh) {
  static_assert(NT >= 64 && NT <= 1024 && NT % 64 == 0, "block of whole waves");
  constexpr int ROUNDS = 8;  // slots per compaction tile
  static_assert(EPT % ROUNDS == 0 || EPT < ROUNDS, "whole tiles of slots");
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  // every load of the slots in use is issued before the first is waited for
  // (loads under a per-lane condition would each be waited for at once):
  // lanes past n load the last score and ignore it
  const int nslot = (n + NT - 1) / NT;  // slots in use, uniform
  float v[EPT];
#pragma unroll
  for (int j = 0; j < EPT; ++j)
    if (j < nslot) v[j] = score[min(j * NT + tid, n - 1)];
  uint32_t key[EPT];
#pragma unroll
  for (int j = 0; j < EPT; ++j) key[j] = j < nslot && j * NT + tid < n ? order_key(v[j]) : 0u;
  // the bits every key shares need no pass: the AND and OR of the keys
  // over the block give the highest bit in which two keys differ, and the
  // passes start there (scores of a few octaves share their sign and high
  // exponent bits, and their first pass would otherwise put most of its
  // counts on a few bins)
  constexpr int NW = NT / 64;
  uint32_t kand = 0xffffffffu, kor = 0u;
#pragma unroll
  for (int j = 0; j < EPT; ++j)
    if (j < nslot && j * NT + tid < n) {
      kand &= key[j];
      kor |= key[j];
    }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    kand &= (uint32_t)__shfl_xor((int)kand, off);
    kor |= (uint32_t)__shfl_xor((int)kor, off);
  }
  if (lane == 0) {  // sh.cnt is free until the compaction, after the passes' barriers
    sh.cnt[0][wid] = kand;
    sh.cnt[0][NW + wid] = kor;
  }
  for (int i = tid; i < 256; i += NT) sh.hist[0][i] = 0;
  __syncthreads();
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    kand &= sh.cnt[0][w];
    kor |= sh.cnt[0][NW + w];
  }
  const uint32_t diff = kand ^ kor;
  const int top = diff ? 31 - __clz((int)diff) : -1;  // highest differing bit
  uint32_t mask = top < 0 ? 0xffffffffu : top == 31 ? 0u : ~((2u << top) - 1u);
  uint32_t prefix = kand & mask, need = (uint32_t)k;
  for (int pass = 0; top - 8 * pass >= 0; ++pass) {
    // digit bits top - 8 pass .. top - 8 pass - 7; the last digit may reach
    // below bit 0 and is then taken from bit 0 (its upper bits are resolved
    // and equal for every candidate)
    const int shift = max(top - 7 - 8 * pass, 0);
    uint32_t* h = sh.hist[pass % 3];
    if (top - 8 * (pass + 1) >= 0)
      for (int i = tid; i < 256; i += NT) sh.hist[(pass + 1) % 3][i] = 0;
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
      if (j * NT >= n) break;  // uniform
      const bool in = j * NT + tid < n;
      hist_add(h, in && (key[j] & mask) == prefix, (key[j] >> shift) & 255u, lane);
    }
    __syncthreads();
    uint32_t c[4], sum = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      c[q] = h[255 - 4 * lane - q];
      sum += c[q];
    }
    uint32_t before = wave_inclusive_scan(sum) - sum;
    int hit = 0;
    uint32_t hit_above = 0;
    bool found = false;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (!found && before < need && before + c[q] >= need) {
        found = true;
        hit = q;
        hit_above = before;
      }
      before += c[q];
    }
    const int src = __ffsll((unsigned long long)__ballot(found)) - 1;
    const uint32_t digit = (uint32_t)__builtin_amdgcn_readlane(255 - 4 * lane - hit, src);
    const uint32_t above = (uint32_t)__builtin_amdgcn_readlane((int)hit_above, src);
    const uint32_t in_bin = (uint32_t)__builtin_amdgcn_readlane((int)pick4(c, hit), src);
    prefix |= digit << shift;
    mask |= 255u << shift;
    need -= above;
    if (need == in_bin) break;  // uniform: the whole bin is taken
  }
  // ordered compaction, tiles of ROUNDS slots (as block_select_topk)
  constexpr int NE = ROUNDS * NW;
  static_assert(NE <= 256, "count scan: at most four entries per lane");
  uint32_t gt_base = 0, eq_base = 0;
#pragma unroll
  for (int t = 0; t < (EPT + ROUNDS - 1) / ROUNDS; ++t) {
    const int base = t * ROUNDS * NT;
    if (base >= n) break;  // uniform
    uint64_t gtm[ROUNDS], eqm[ROUNDS];
    uint32_t mine = 0;
#pragma unroll
    for (int j = 0; j < ROUNDS; ++j) {
      const int slot = t * ROUNDS + j;
      bool gt = false, eq = false;
      if (slot < EPT && base + j * NT + tid < n) {
        const uint32_t km = key[slot < EPT ? slot : 0] & mask;
        gt = km > prefix;
        eq = km == prefix;
      }
      gtm[j] = __ballot(gt);
      eqm[j] = __ballot(eq);
      if (lane == j) mine = ((uint32_t)__popcll(gtm[j]) << 16) | (uint32_t)__popcll(eqm[j]);
    }
    uint32_t* cnt = sh.cnt[t & 1];
    if (lane < ROUNDS) cnt[lane * NW + wid] = mine;
    __syncthreads();
    uint32_t c[4], sum = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * lane + q;
      c[q] = e < NE ? cnt[e] : 0u;
      sum += c[q];
    }
    const uint32_t incl = wave_inclusive_scan(sum);
    const uint32_t total = (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
    uint32_t ex[4];
    ex[0] = incl - sum;
#pragma unroll
    for (int q = 1; q < 4; ++q) ex[q] = ex[q - 1] + c[q - 1];
#pragma unroll
    for (int j = 0; j < ROUNDS; ++j) {
      if (base + j * NT >= n) break;  // uniform
      const int e = j * NW + wid;
      const int q = e & 3;
      const uint32_t pick = q == 0 ? ex[0] : q == 1 ? ex[1] : q == 2 ? ex[2] : ex[3];
      const uint32_t off = (uint32_t)__builtin_amdgcn_readlane((int)pick, e >> 2);
      const uint64_t gm = gtm[j], em = eqm[j];
      const bool gt = (gm >> lane) & 1ull, eq = (em >> lane) & 1ull;
      const uint32_t gt_before = gt_base + (off >> 16) +
          __builtin_amdgcn_mbcnt_hi((uint32_t)(gm >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)gm, 0u));
      const uint32_t eq_before = eq_base + (off & 0xffffu) +
          __builtin_amdgcn_mbcnt_hi((uint32_t)(em >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)em, 0u));
      if (gt || (eq && eq_before < need)) {
        const uint32_t pos = gt_before + min(eq_before, need);
        if (pos < (uint32_t)k) emit(pos, base + j * NT + tid);
      }
    }
    gt_base += total >> 16;
    eq_base += total & 0xffffu;
  }
}

// Top-k by whichever form fits: registers for n <= EPT * NT, else the
// general loop over `score`.
template <int NT, int EPT, typename Emit>
__device__ __forceinline__ void block_select_topk_any(const float* score, int n, int k, Emit emit,
                                                      SelectShared<NT>& sh) {
  if (n <= EPT * NT)
    block_select_topk_regs<NT, EPT>(score, n, k, emit, sh);
  else
    block_select_topk<NT>(score, n, k, emit, sh);
}

// ------------------------------------------------------------ LDS staging

// Rows of D elements moved to LDS in 16-byte vectors, row stride D plus one
// vector of padding.  Vector v of a chunk is (row v / VPR, column v % VPR);
// thread t owns vectors t, t + NT, ...  Loads go to registers first (all of a
// thread's loads in flight together), then to LDS, so a chunk can be
// prefetched while the previous one is consumed.
template <typename T, int D, int ROWS, int NT>
struct RowStager {
  static constexpr int EPV = 16 / sizeof(T);
  static constexpr int VPR = D / EPV;
  static constexpr int STRIDE = D + EPV;
  static constexpr int PER_THREAD = (ROWS * VPR + NT - 1) / NT;
  u32x4 buf[PER_THREAD];

  // src(r) -> row pointer, or nullptr for a zero row; r < ROWS
  template <class Src>
  __device__ __forceinline__ void load(Src src) {
    const T* rowp[PER_THREAD];
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int v = i * NT + threadIdx.x;
      rowp[i] = v < ROWS * VPR ? src(v / VPR) : nullptr;
    }
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int v = i * NT + threadIdx.x;
      buf[i] = rowp[i] ? *reinterpret_cast<const u32x4*>(rowp[i] + (v % VPR) * EPV)
                       : u32x4{0u, 0u, 0u, 0u};
    }
  }

  __device__ __forceinline__ void store(T* dst) const {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int v = i * NT + threadIdx.x;
      if (v < ROWS * VPR)
        *reinterpret_cast<u32x4*>(dst + (v / VPR) * STRIDE + (v % VPR) * EPV) = buf[i];
    }
  }

  // bf16 only: store transposed, dst[c * TSTRIDE + r] = row r, channel c
  template <int TSTRIDE>
  __device__ __forceinline__ void store_transposed(uint16_t* dst) const {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int v = i * NT + threadIdx.x;
      if (v < ROWS * VPR) {
        const int r = v / VPR, c0 = (v % VPR) * 8;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          dst[(c0 + 2 * e) * TSTRIDE + r] = (uint16_t)(buf[i][e] & 0xffffu);
          dst[(c0 + 2 * e + 1) * TSTRIDE + r] = (uint16_t)(buf[i][e] >> 16);
        }
      }
    }
  }
};

// Copies `rows` (runtime, any count) rows to LDS, 8 loads in flight per
// thread; src(r) -> row pointer.
template <typename T, int D, int NT, class Src>
__device__ __forceinline__ void stage_rows_any(T* dst, int rows, Src src) {
  constexpr int EPV = 16 / sizeof(T);
  constexpr int VPR = D / EPV;
  constexpr int STRIDE = D + EPV;
  constexpr int BATCH = 8;
  const int total = rows * VPR;
  for (int base = 0; base < total; base += BATCH * NT) {
    u32x4 buf[BATCH];
#pragma unroll
    for (int i = 0; i < BATCH; ++i) {
      const int v = base + i * NT + threadIdx.x;
      buf[i] = v < total ? *reinterpret_cast<const u32x4*>(src(v / VPR) + (v % VPR) * EPV)
                         : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < BATCH; ++i) {
      const int v = base + i * NT + threadIdx.x;
      if (v < total)
        *reinterpret_cast<u32x4*>(dst + (v / VPR) * STRIDE + (v % VPR) * EPV) = buf[i];
    }
  }
}

// ------------------------------------------------------------ async LDS fill
//
// gfx950 loads 16 bytes per lane straight from global memory into LDS
// (global_load_lds_dwordx4): lane l's bytes land at M0 + 16 l.  The load is
// issued through inline asm so that the compiler does not drain every
// outstanding load before each LDS read; the code waits explicitly with
// wait_vmcnt_chunks(), which is exact because vector-memory operations
// complete in issue order.  Between issue and wait a wave issues no other
// vector-memory operation.

__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)p;
}

// M0 is saved and restored inside the statement: the compiler may keep a
// value of its own there.  STREAM marks data read exactly once (the `nt`
// cache policy): it then does not displace data that later kernels re-read.
template <bool STREAM = false>
__device__ __forceinline__ void async_load16(const void* g, uint32_t lds_byte) {
  uint32_t saved;
  if constexpr (STREAM)
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off nt\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(g), "s"(lds_byte)
        : "memory");
  else
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(g), "s"(lds_byte)
        : "memory");
}

// Workgroup barrier for LDS traffic only: waits for this wave's LDS
// operations, not for outstanding global loads.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until at most k * IPW vector-memory operations of this wave are
// outstanding (k = chunks allowed to remain in flight, 0..3).
template <int IPW>
__device__ __forceinline__ void wait_vmcnt_chunks(int k) {
  static_assert(3 * IPW <= 63, "vmcnt field is 6 bits");
  switch (k) {
    case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    case 1: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(IPW) : "memory"); break;
    case 2: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * IPW) : "memory"); break;
    default: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(3 * IPW) : "memory"); break;
  }
}

// Rows of G 16-byte granules stored unpadded in LDS; granule k of row r
// lives in slot k ^ swz(r).  For the access patterns below (16 rows at one
// granule; rows 8(m/4)+m%4 of a 32-row block) the slots, hence the banks,
// differ across the 16 lanes that share a lane group.
template <int G>
__device__ __forceinline__ int granule_swz(int r) {
  if constexpr (G >= 16) return (r & 15) ^ (((r >> 4) & 1) << 2);
  return ((r >> 1) & 7) ^ (((r >> 4) & 1) << 1);
}

template <int G>
__device__ __forceinline__ int granule_offset(int r, int k) {
  return r * (16 * G) + 16 * (k ^ granule_swz<G>(r));
}

// Queues one chunk of CR rows (G granules each) into LDS at lds_base:
// instruction i of wave w fills bytes [1024 (w IPW + i), +1024), i.e. rows
// (w IPW + i) 64/G .. +64/G.  rowptr(r) returns a valid global row address
// for every r < CR (callers clamp rows past their range).
template <int CR, int G, int NW, bool STREAM = false, class RowPtr>
__device__ __forceinline__ void issue_chunk(uint32_t lds_base, const RowPtr& rowptr) {
  constexpr int RPI = 64 / G;
  constexpr int IPW = CR * G / (64 * NW);
  static_assert(IPW * 64 * NW == CR * G, "chunk must fill whole instructions");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < IPW; ++i) {
    const int inst = wave * IPW + i;
    const int r = inst * RPI + lane / G;
    const int k = (lane % G) ^ granule_swz<G>(r);
    const unsigned char* g = reinterpret_cast<const unsigned char*>(rowptr(r)) + 16 * k;
    async_load16<STREAM>(g, __builtin_amdgcn_readfirstlane(lds_base + 1024u * inst));
  }
}

// ------------------------------------------------------------ launch shape

// Maps the hardware workgroup id to a logical id so that consecutive logical
// ids run on the same XCD (workgroups are dealt round-robin over the 8 XCDs).
__device__ __forceinline__ int xcd_swizzle(int bid, int nblocks) {
  if ((nblocks & 7) != 0) return bid;
  return (bid & 7) * (nblocks >> 3) + (bid >> 3);
}

}  // namespace wf
