// Token-level skim for bf16 keys and a query block of at most 64 rows: the
// Haar wavelet at 3..5 levels (token_skim_kernel) and Daubechies-2 at 6
// levels (token_db2_kernel, further below).
//
// The Haar approximation of block j at level J is 2^{-J/2} times the sum of
// its 2^J keys (eq. 5 with the Haar filter, applied J times), and the skim
// logit is linear in the key, so the coarse logit of eq. 7 is the scaled sum
// of the block's token logits:  l_qj = 2^{-J/2} sum_{t in block j} s_qt,
// s_qt = scale <Q_q, K_t>.  One pass over the keys therefore computes every
// token logit on bf16 MFMA and reduces it per block to
//   * the coarse logit l_qj                        (input of eqs. 7-8)
//   * the block log-sum-exp  e_qj = log sum_{t in block j} exp(s_qt)
// stored per block as a row of B coarse logits followed by a row of B
// log-sum-exps ([U][nJ][2][B]).
// The second gives the softmax normalisers of the token scan over the
// selected pool (Section 3.2) without a separate pass over the pool:
//   M_q = max_{j in seg} e_qj,   Z_q = sum_{j in seg} exp(e_qj - M_q),
// with M_q at or above every pool logit of query q.
//
// The same kernel without the log-sum-exps serves the scales b <= 5 of the
// multi-scale recursion (Alg. 1): it writes only the coarse logits,
// query-major ([U][B][nJ], the layout of the coefficient tiles), and the
// per-range statistics, over all keys at the first scale and over the
// gathered kept blocks below it.
//
// The keys stream through an LDS ring filled by direct global->LDS loads;
// see token_skim_kernel for the roles of its waves.
#include "wf_device.hpp"
#include "wf_kernels.hpp"
#include "wf_launch.hpp"

#include <mutex>

namespace wf {

// one value joins a running (max, sum of exp) pair
__device__ __forceinline__ void stat_add(float& m, float& z, float x) {
  if (x > m) {
    z = z * __expf(m - x) + 1.f;
    m = x;
  } else {
    z += __expf(x - m);
  }
}

// Workgroup of the token-level skim: 8 waves, wave w scores the 32-token
// slice w % 4 of every 128-token chunk against query rows 32 (w / 4) + 0..31.
// The keys are read exactly once and are loaded with the streaming (nt)
// policy, which keeps them from evicting the block rows before those leave.
// Every wave puts its block results into an LDS batch laid out as the
// global array; waves 0..3 issue every ring load and store nothing to global
// memory, waves 4..7 issue no loads and copy each finished batch out as one
// contiguous run.  (Stores count in the same per-wave counter as the ring
// loads, so a loading wave that also stored would wait for its stores at
// every ring wait; and few long write runs interleave with the key stream
// more cheaply than many short ones.)
constexpr int kTokBlock = 512;

// Lane l of a wave holds, after the 32x32x16 products of its slice, the
// logits of query 32 (w / 4) + l % 32 with the slice's tokens
//   8 (v / 4) + 4 (l / 32) + v % 4,   v < 16,
// so block b (of 2^J tokens, J = 3, 4, 5) of the slice is the lane's values
// v in [b 2^J / 2, (b + 1) 2^J / 2) together with the same values of lane
// l ^ 32.  Each lane keeps NST of the slice's 32 / 2^J blocks: block 0 in the
// lanes l < 32 (J = 5), block l / 32 (J = 4), blocks 2 (l / 32) + n, n < 2
// (J = 3).
template <int J>
struct SliceBlocks {
  static constexpr int NBLK = 32 >> J;         // blocks per slice
  static constexpr int VPB = 16 / NBLK;        // lane values per block
  static constexpr int NST = J == 3 ? 2 : 1;   // blocks kept per lane
  static constexpr int BPC = 128 >> J;         // blocks per 128-token chunk
  static constexpr int BATCH = J == 5 ? 2 : 1;  // chunks per LDS batch (4 or 8 KiB at 64 queries)
  __device__ static int block(int n, int hi) { return J == 5 ? 0 : J == 4 ? hi : 2 * hi + n; }
  __device__ static bool keeps(int hi) { return J != 5 || hi == 0; }
};

// Blocks of 2 or 4 tokens (J = 1, 2) lie inside one lane: its values
// v in [i 2^J, (i + 1) 2^J) are the block (8 (v / 4) + 4 (l / 32) + v % 4) >> J
// of the slice, 16 / 2^J of them per lane.
//
// Chunks per LDS batch.  With the log-sum-exps a batch holds block rows of
// 2 B floats; without them it holds NBB = 32 or 64 blocks of every query row
// (a run of 128 bytes or more per row), block e of row q at column
// e ^ (q mod NBB), so that the 32 query rows a wave writes at once fall in
// distinct banks.
template <int J, bool LSE>
constexpr int token_batch_chunks() {
  return LSE ? SliceBlocks<J>::BATCH : ((128 >> J) >= 32 ? 1 : 32 / (128 >> J));
}

// LDS bytes of one token-skim batch slot
template <int J, bool LSE>
constexpr size_t token_batch_bytes(int B) {
  constexpr int nbb = token_batch_chunks<J, LSE>() * (128 >> J);
  return (size_t)nbb * (LSE ? 2 * B : B) * sizeof(float);
}

// Waves per SIMD the token skim is compiled to allow: four lets two
// workgroups share a CU; with 128-wide keys, the 8-token blocks with their
// log-sum-exps and the 2-token blocks need more registers than that leaves,
// and run one workgroup per CU.
constexpr int token_skim_waves_per_simd(int D, int J, bool lse) {
  return D == 128 && ((lse && J == 3) || (!lse && J == 1)) ? 2 : 4;
}

template <int D, int J, bool LSE, bool GATHER = false>
__global__ __launch_bounds__(kTokBlock, token_skim_waves_per_simd(D, J, LSE)) void token_skim_kernel(
    TokenSkimArgs a) {
  constexpr int NW = kTokBlock / kWave;  // 8
  constexpr int NIW = NW / 2;            // loading waves
  constexpr int CR = kScanChunk;         // tokens per chunk
  constexpr int G = D / 8;               // 16-byte granules per key row
  constexpr int CHB = CR * 2 * D;
  constexpr int IPW = CR * G / (64 * NIW);
  constexpr int KS = D / 16;             // k-steps of the 32x32x16 product
  using SB = SliceBlocks<J>;
  constexpr int BPC = 128 >> J;                           // blocks per chunk
  constexpr int BATCH = token_batch_chunks<J, LSE>();
  constexpr int NBB = BATCH * BPC;                        // blocks per batch
  static_assert(J >= 1 && J <= 5, "blocks of 2 .. 32 tokens");
  static_assert(!LSE || J >= 3, "log-sum-exps for blocks of 8, 16 or 32 tokens");
  static_assert(!(LSE && GATHER), "gathered rows only without the log-sum-exps");
  static_assert(CR == 32 * NIW, "four 32-token slices per chunk");
  const int B = a.B;
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* ring = smem;  // [nbuf][CHB]
  // two slots: [NBB][2][B] coarse logits, then log-sum-exps (LSE), or
  // [B][NBB] coarse logits (columns swizzled)
  float* batch = reinterpret_cast<float*>(smem + (size_t)a.nbuf * CHB);
  // [NW][32][2] running pairs, merged after the last ring load has landed:
  // they reuse the ring's first bytes
  float* red = reinterpret_cast<float*>(smem);
  const int slot_floats = LSE ? NBB * 2 * B : B * NBB;

  const int item = xcd_swizzle(blockIdx.x, gridDim.x);
  const int u = item / a.R, r = item % a.R;
  const long tb = (long)r * a.span;
  const long te = min(tb + (long)a.span, (long)a.L);
  const int nch = (int)((te - tb + CR - 1) / CR);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ts = wave & 3, qt = wave >> 2;
  const bool loader = qt == 0;
  const int hi = lane >> 5, col = lane & 31;
  const int q = 32 * qt + col;
  const bool live = 32 * qt < B;  // wave-uniform: this query tile has rows

  const bf16_t* qrow = reinterpret_cast<const bf16_t*>(a.Q) + ((long)u * B + min(q, B - 1)) * D;
  u32x4 qreg[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) qreg[s] = *reinterpret_cast<const u32x4*>(qrow + 16 * s + 8 * hi);
  // the query operand is consumed here, before any ring load is queued, so
  // that no wait for it lands inside the ring loop
#pragma unroll
  for (int s = 0; s < KS; ++s) asm volatile("" ::"v"(qreg[s]));

  // row r of the chunk at c0: key row c0 + r, or on a refinement scale
  // gathered row p = c0 + r, token par[p >> pshift] 2^pshift + p mod 2^pshift
  // (rows past the range repeat its last row; ids are clamped into the unit)
  struct Rows {
    const bf16_t* Kunit;
    const int32_t* par;  // LDS: the range's parent ids from p_lo on, or null
    long c0, tlast;
    int pshift, p_lo, last;
    __device__ __forceinline__ const bf16_t* operator()(int r) const {
      const long p = min(c0 + r, tlast);
      if (!par) return Kunit + p * D;
      const int t = (par[(int)(p >> pshift) - p_lo] << pshift) | (int)(p & ((1 << pshift) - 1));
      return Kunit + (long)min(max(t, 0), last) * D;
    }
  } rows{reinterpret_cast<const bf16_t*>(a.K) + (long)u * a.Ls * D, nullptr, tb, te - 1,
         a.pshift, (int)(tb >> a.pshift), (int)a.Ls - 1};
  if constexpr (GATHER) {
    {
      // stage the range's parent ids (every thread reads them back below)
      int32_t* par_sh = reinterpret_cast<int32_t*>(batch + 2 * slot_floats);
      const int n_ids = (int)((te - 1) >> a.pshift) - rows.p_lo + 1;
      const int32_t* src = a.parent + (long)u * a.npar + rows.p_lo;
      for (int i = threadIdx.x; i < n_ids && i < a.par_cap; i += kTokBlock) par_sh[i] = src[i];
      __syncthreads();
      rows.par = par_sh;
    }
  }
  const uint32_t ring_lds = lds_offset(ring);
  const int nbuf = a.nbuf;
  // the keys, and the gathered rows of a refinement scale, stream past the
  // caches (for the gathered rows that measured faster than cached loads,
  // although the attention reads many of them again)
  auto issue_rows = [&](uint32_t slot) { issue_chunk<CR, G, NIW, true>(slot, rows); };
  if (loader) {
    for (int k = 0; k < nch && k < nbuf - 1; ++k) {
      rows.c0 = tb + (long)k * CR;
      issue_rows(ring_lds + (uint32_t)(k * CHB));
    }
  }

  const long jend = te >> J;                        // blocks of this range end here
  const float cl = a.scale * a.norm;

  // waves 4..7: copy batch k (its blocks inside the range) to global memory
  auto copy_batch = [&](int k) {
    const long jb0 = (tb >> J) + (long)k * NBB;
    const int nb = (int)min((long)NBB, jend - jb0);
    const float* src = batch + (k & 1) * slot_floats;
    const int t = (wave - NIW) * 64 + lane;
    if constexpr (LSE) {
      // one contiguous run of nb block rows ([nJ][2][B])
      const int nf = nb * 2 * B;
      float* dst = a.blocks + ((long)u * a.nJ + jb0) * 2 * B;
      if ((B & 1) == 0) {  // block rows are 16-byte multiples
        for (int i = t; i < nf / 4; i += NIW * 64)
          reinterpret_cast<float4*>(dst)[i] = reinterpret_cast<const float4*>(src)[i];
      } else {
        for (int i = t; i < nf; i += NIW * 64) dst[i] = src[i];
      }
    } else {
      // one run of nb logits per query row ([B][nJ]); NBB is a power of two
      // (no integer division in the index)
      float* dst = a.blocks + (long)u * B * a.nJ + jb0;
      constexpr int LNB = NBB == 32 ? 5 : 6;
      static_assert((1 << LNB) == NBB, "32 or 64 blocks a batch");
      if (J == 1 && nb == NBB && (a.nJ & 3) == 0) {
        // a whole batch of 2-token blocks: four adjacent logits of a row per
        // 16-byte store (jb0 is a multiple of 64)
        constexpr int F = NBB / 4, LF = LNB - 2;
        for (int i = t; i < F * B; i += NIW * 64) {
          const int qq = i >> LF, e0 = 4 * (i & (F - 1)), x = qq & (NBB - 1);
          const float* row = src + qq * NBB;
          const float4 o = make_float4(row[e0 ^ x], row[(e0 + 1) ^ x], row[(e0 + 2) ^ x],
                                       row[(e0 + 3) ^ x]);
          *reinterpret_cast<float4*>(dst + (long)qq * a.nJ + e0) = o;
        }
      } else {
        for (int i = t; i < NBB * B; i += NIW * 64) {
          const int qq = i >> LNB, e = i & (NBB - 1);
          if (e < nb) dst[(long)qq * a.nJ + e] = src[qq * NBB + (e ^ (qq & (NBB - 1)))];
        }
      }
    }
  };

  float cm = -INFINITY, cz = 0.f;  // running max / sum of exp of the kept coarse logits
  for (int ch = 0; ch < nch; ++ch) {
    const long c0 = tb + (long)ch * CR;
    if (loader) wait_vmcnt_chunks<IPW>(min(nch - 1 - ch, nbuf - 2));
    lds_barrier();
    if (loader) {
      if (ch + nbuf - 1 < nch) {
        rows.c0 = tb + (long)(ch + nbuf - 1) * CR;
        issue_rows(ring_lds + (uint32_t)(((ch + nbuf - 1) % nbuf) * CHB));
      }
    } else if (ch > 0 && ch % BATCH == 0) {
      copy_batch(ch / BATCH - 1);
    }
    const long slice0 = c0 + 32 * ts;
    if (!live || slice0 >= te) continue;  // uniform per wave; no barrier follows
    const unsigned char* buf = ring + (ch % nbuf) * CHB;
    const int row = 32 * ts + col;
    f32x16 acc = {};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const u32x4 ka = *reinterpret_cast<const u32x4*>(buf + granule_offset<G>(row, 2 * s + hi));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, ka),
                                                    __builtin_bit_cast(bf16x8, qreg[s]), acc, 0, 0, 0);
    }
    float* slot = batch + ((ch / BATCH) & 1) * slot_floats;
    const int bl0 = (ch % BATCH) * BPC + ((32 * ts) >> J);  // slice's first block in the batch
    if constexpr (J <= 2) {
      // every block lies in one lane
      constexpr int VPB = 1 << J, NL = 16 / VPB;
      if constexpr (J == 1) {
        // eight logits a lane: their maximum first, then one rescale of the
        // running pair and a term each (no branch per logit)
        float lv[NL];
        float bmx = -INFINITY;
#pragma unroll
        for (int i = 0; i < NL; ++i) {
          const int b = (8 * ((i * VPB) / 4) + 4 * hi + (i * VPB) % 4) >> J;
          lv[i] = (acc[2 * i] + acc[2 * i + 1]) * cl;
          if (q < B && (slice0 >> J) + b < jend) {
            bmx = fmaxf(bmx, lv[i]);
            slot[q * NBB + ((bl0 + b) ^ (q & (NBB - 1)))] = lv[i];
          } else {
            lv[i] = -INFINITY;
          }
        }
        if (bmx > -INFINITY) {
          const float mn = fmaxf(cm, bmx);
          float zz = cz * __expf(cm - mn);
#pragma unroll
          for (int i = 0; i < NL; ++i) zz += __expf(lv[i] - mn);
          cm = mn;
          cz = zz;
        }
      } else {
#pragma unroll
        for (int i = 0; i < NL; ++i) {
          float s_ = 0.f;
#pragma unroll
          for (int v = i * VPB; v < (i + 1) * VPB; ++v) s_ += acc[v];
          const int b = (8 * ((i * VPB) / 4) + 4 * hi + (i * VPB) % 4) >> J;
          const float l = s_ * cl;
          if (q < B && (slice0 >> J) + b < jend) {
            stat_add(cm, cz, l);
            slot[q * NBB + ((bl0 + b) ^ (q & (NBB - 1)))] = l;
          }
        }
      }
    } else {
      constexpr int NBLK = SB::NBLK, VPB = SB::VPB, NST = SB::NST;
      const float c2 = a.scale * kLog2e;
      // raw block sums (and maxima), completed with the partner lane l ^ 32
      float bs[NBLK], bm[NBLK], be[NBLK];
#pragma unroll
      for (int b = 0; b < NBLK; ++b) {
        bs[b] = 0.f;
        bm[b] = -INFINITY;
#pragma unroll
        for (int v = b * VPB; v < (b + 1) * VPB; ++v) {
          bs[b] += acc[v];
          if constexpr (LSE) bm[b] = fmaxf(bm[b], acc[v]);
        }
        bs[b] = add_xor32(bs[b]);
        be[b] = 0.f;
        if constexpr (LSE) {
          bm[b] = max_xor32(bm[b]);
          const float off = -bm[b] * c2;
#pragma unroll
          for (int v = b * VPB; v < (b + 1) * VPB; ++v) be[b] += __builtin_amdgcn_exp2f(fmaf(acc[v], c2, off));
          be[b] = add_xor32(be[b]);
        }
      }
      const bool keeps = SB::keeps(hi);
#pragma unroll
      for (int n = 0; n < NST; ++n) {
        const int b = SB::block(n, hi);
        // b takes at most two values across the wave: select, do not index
        float s_ = bs[0], m_ = bm[0], e_ = be[0];
#pragma unroll
        for (int k = 1; k < NBLK; ++k)
          if (b == k) {
            s_ = bs[k];
            m_ = bm[k];
            e_ = be[k];
          }
        const float l = s_ * cl;
        if (keeps && q < B && (slice0 >> J) + b < jend) {
          stat_add(cm, cz, l);
          if constexpr (LSE) {
            slot[(bl0 + b) * 2 * B + q] = l;
            slot[((bl0 + b) * 2 + 1) * B + q] = fmaf(m_, a.scale, __logf(e_));
          } else {
            slot[q * NBB + ((bl0 + b) ^ (q & (NBB - 1)))] = l;
          }
        }
      }
    }
  }
  __syncthreads();  // the last batch is complete in LDS
  if (!loader) copy_batch((nch - 1) / BATCH);

  // merge the running coarse statistics: partner lanes, then the four
  // slices of the query tile
  {
    const float m2 = partner32(cm), z2 = partner32(cz);
    stat_absorb(cm, cz, m2, z2);
  }
  if (hi == 0) {
    red[(wave * 32 + col) * 2] = cm;
    red[(wave * 32 + col) * 2 + 1] = cz;
  }
  __syncthreads();
  float* ws = a.wstats + ((long)u * a.R + r) * 2 * B;
  for (int qq = threadIdx.x; qq < B; qq += kTokBlock) {
    const int t = qq >> 5, c = qq & 31;
    float mx = -INFINITY, z = 0.f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int w = 4 * t + k;
      stat_absorb(mx, z, red[(w * 32 + c) * 2], red[(w * 32 + c) * 2 + 1]);
    }
    ws[qq] = mx;
    ws[B + qq] = z;
  }
}

// Blocks of 32 tokens with their log-sum-exps, one workgroup per CU: the
// same products and block reductions as token_skim_kernel<D, 5, true>, but
// every wave keeps its block results in registers and stores them only after
// the range's last key load has landed.  Writes issued while the key stream
// runs cost about four read-byte times per byte written (on one MI355X a
// 1 GiB ring read at 7.25 TB/s slowed from 148 to 192 us when 64 MiB of
// writes were spread over it, in 4 KiB or 32 KiB batches alike, and to 160 us
// when the same writes followed it), so the results wait until the reads are
// done.  A lane holds one value per chunk (the coarse logit of its query in
// lanes 0..31, the block's log-sum-exp in lanes 32..63), 128 chunks in four
// register vectors of 32, written through a wave-uniform register index;
// that takes the register file of two waves per SIMD, hence one workgroup
// per CU with the ring three chunks deep.
typedef float f32x32 __attribute__((ext_vector_type(32)));
constexpr int kHeldChunks = 128;

template <int D>
__global__ __launch_bounds__(kTokBlock, 2) void token_skim_held_kernel(TokenSkimArgs a) {
  constexpr int NIW = kTokBlock / kWave / 2;  // loading waves
  constexpr int CR = kScanChunk;
  constexpr int G = D / 8;
  constexpr int CHB = CR * 2 * D;
  constexpr int IPW = CR * G / (64 * NIW);
  constexpr int KS = D / 16;
  constexpr int J = 5;
  static_assert(CR == 32 * NIW, "four 32-token slices (one block each) per chunk");
  const int B = a.B;
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* ring = smem;                   // [nbuf][CHB]
  float* red = reinterpret_cast<float*>(smem);  // [8][32][2] once the ring is idle

  const int item = xcd_swizzle(blockIdx.x, gridDim.x);
  const int u = item / a.R, r = item % a.R;
  const long tb = (long)r * a.span;
  const long te = min(tb + (long)a.span, (long)a.L);
  const int nch = (int)((te - tb + CR - 1) / CR);  // at most kHeldChunks (host-checked)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ts = wave & 3, qt = wave >> 2;
  const bool loader = qt == 0;
  const int hi = lane >> 5, col = lane & 31;
  const int q = 32 * qt + col;
  const bool live = 32 * qt < B;  // wave-uniform: this query tile has rows

  const bf16_t* qrow = reinterpret_cast<const bf16_t*>(a.Q) + ((long)u * B + min(q, B - 1)) * D;
  u32x4 qreg[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) qreg[s] = *reinterpret_cast<const u32x4*>(qrow + 16 * s + 8 * hi);
#pragma unroll
  for (int s = 0; s < KS; ++s) asm volatile("" ::"v"(qreg[s]));

  // row r of the chunk at c0 (rows past the range repeat its last row)
  struct Rows {
    const bf16_t* Kunit;
    long c0, tlast;
    __device__ __forceinline__ const bf16_t* operator()(int r) const {
      return Kunit + min(c0 + r, tlast) * D;
    }
  } rows{reinterpret_cast<const bf16_t*>(a.K) + (long)u * a.Ls * D, tb, te - 1};
  const uint32_t ring_lds = lds_offset(ring);
  const int nbuf = a.nbuf;
  if (loader) {
    for (int k = 0; k < nch && k < nbuf - 1; ++k) {
      rows.c0 = tb + (long)k * CR;
      issue_chunk<CR, G, NIW, true>(ring_lds + (uint32_t)(k * CHB), rows);
    }
  }
  const long jend = te >> J;
  const float cl = a.scale * a.norm;
  const float c2 = a.scale * kLog2e;
  float cm = -INFINITY, cz = 0.f;  // running max / sum of exp of the coarse logits

  // chunk ch: the lane's held value (coarse logit or block log-sum-exp)
  auto step = [&](int ch) -> float {
    if (loader) wait_vmcnt_chunks<IPW>(min(nch - 1 - ch, nbuf - 2));
    lds_barrier();  // chunk ch visible; everyone is past chunk ch - 1
    if (loader && ch + nbuf - 1 < nch) {
      rows.c0 = tb + (long)(ch + nbuf - 1) * CR;
      issue_chunk<CR, G, NIW, true>(ring_lds + (uint32_t)(((ch + nbuf - 1) % nbuf) * CHB), rows);
    }
    const long slice0 = tb + (long)ch * CR + 32 * ts;
    if (!live || slice0 >= te) return 0.f;  // uniform per wave; never stored
    const unsigned char* buf = ring + (ch % nbuf) * CHB;
    const int row = 32 * ts + col;
    f32x16 acc = {};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const u32x4 ka = *reinterpret_cast<const u32x4*>(buf + granule_offset<G>(row, 2 * s + hi));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, ka),
                                                    __builtin_bit_cast(bf16x8, qreg[s]), acc, 0, 0, 0);
    }
    // the lane's 16 logits and those of lane l ^ 32 are the slice's block
    float bs = 0.f, bm = -INFINITY;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      bs += acc[v];
      bm = fmaxf(bm, acc[v]);
    }
    bs = add_xor32(bs);
    bm = max_xor32(bm);
    const float off = -bm * c2;
    float be = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) be += __builtin_amdgcn_exp2f(fmaf(acc[v], c2, off));
    be = add_xor32(be);
    const float l = bs * cl;
    if (hi == 0 && q < B && (slice0 >> J) < jend) stat_add(cm, cz, l);
    return hi ? fmaf(bm, a.scale, __logf(be)) : l;
  };
  f32x32 h0, h1, h2, h3;
#define WF_HELD_GROUP(g, hv)                          \
  for (int i = 0; i < 32; ++i) {                      \
    const int ch = 32 * (g) + i;                      \
    if (ch >= nch) break;                             \
    hv[__builtin_amdgcn_readfirstlane(i)] = step(ch); \
  }
  WF_HELD_GROUP(0, h0)
  WF_HELD_GROUP(1, h1)
  WF_HELD_GROUP(2, h2)
  WF_HELD_GROUP(3, h3)
#undef WF_HELD_GROUP
  __syncthreads();  // every ring read is done: its first bytes take the pairs below

  // block rows [nJ][2][B]: in chunk ch, wave (ts, qt) holds block
  // j0 + 4 ch (j0 = tb / 32 + ts), lane l its row 2 j + hi at column q, so
  // consecutive chunks are 8 B floats apart; the chunks whose block ends
  // inside the range are the first nv (wave-uniform).  The addresses are one
  // add apart: with per-store index arithmetic the dependent 64-bit products
  // held the write phase back.
  const long j0 = (tb >> J) + ts;
  const int nv = __builtin_amdgcn_readfirstlane(
      (int)max(0L, min((long)nch, (jend - j0 + 3) / 4)));
  if (live && q < B) {
    float* p = a.blocks + ((long)u * a.nJ + j0) * 2 * B + (long)hi * B + q;
    const long stride = 8L * B;
    auto flush = [&](const f32x32& hv, int g) {
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        if (32 * g + i >= nv) break;  // uniform
        p[(long)(32 * g + i) * stride] = hv[i];
      }
    };
    flush(h0, 0);
    flush(h1, 1);
    flush(h2, 2);
    flush(h3, 3);
  }

  // the range's coarse statistics, as token_skim_kernel
  {
    const float m2 = partner32(cm), z2 = partner32(cz);
    stat_absorb(cm, cz, m2, z2);
  }
  if (hi == 0) {
    red[(wave * 32 + col) * 2] = cm;
    red[(wave * 32 + col) * 2 + 1] = cz;
  }
  __syncthreads();
  float* ws = a.wstats + ((long)u * a.R + r) * 2 * B;
  for (int qq = threadIdx.x; qq < B; qq += kTokBlock) {
    const int t = qq >> 5, c = qq & 31;
    float mx = -INFINITY, z = 0.f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int w = 4 * t + k;
      stat_absorb(mx, z, red[(w * 32 + c) * 2], red[(w * 32 + c) * 2 + 1]);
    }
    ws[qq] = mx;
    ws[B + qq] = z;
  }
}

// Daubechies-2 at J = 6 from token logits.  The level-6 approximation is one
// banded filter of the keys (A[n] = sum_m f[m] K[64 n + m], 190 taps), so
// the coarse logit is the same filter over token logits:
//   l_n = P_0(n) + P_1(n + 1) + P_2(n + 2),  P_k(c) = sum_{o < 64} f[64 k + o] s_(64 c + o),
// with s the raw products times the logit scale.  Every slice (32 tokens,
// half a block) forms its three partials and its (max, sum of exp) on the
// lanes of the 32x32 product; they wait in a three-chunk LDS ring until the
// two blocks after theirs are in, and waves 4..7 then add the six partials of
// a coefficient in a fixed order and store its block row (coarse logit, then
// the block's log-sum-exp, as the Haar path).  A range reads one chunk past
// its end (its last coefficients need the next two blocks), wrapped around
// the unit for the periodic extension.  With the symmetric extension the
// last three coefficients of the unit use the end filters E_m instead, from
// their own partials of the last three blocks, which the range owning them
// reads (its reads stop at the unit's end).
//
// HOLD (at most 32 query rows and 128 chunks a range): the block rows wait
// in registers until the range's keys are read, as in token_skim_held_kernel;
// wave 4 + c mod 4 completes the coefficients of chunk c, so that each of
// waves 4..7 holds a coefficient pair every fourth chunk (32 slots of two
// values a lane).
template <int D, bool HOLD = false>
__global__ __launch_bounds__(kTokBlock, 2) void token_db2_kernel(TokenSkimArgs a, Db2TokenTaps tp,
                                                                 int periodic) {
  constexpr int NW = kTokBlock / kWave;  // 8
  constexpr int NIW = NW / 2;            // loading waves
  constexpr int CR = kScanChunk;         // tokens per chunk: two blocks
  constexpr int G = D / 8;
  constexpr int CHB = CR * 2 * D;
  constexpr int IPW = CR * G / (64 * NIW);
  constexpr int KS = D / 16;
  static_assert(CR == 128, "two 64-token blocks per chunk");
  const int B = a.B;
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* ring = smem;                                           // [nbuf][CHB]
  float* part = reinterpret_cast<float*>(smem + (size_t)a.nbuf * CHB);  // [3][4][3][B]
  float* sst = part + 36 * B;                                           // [3][4][2][B]
  float* edg = sst + 24 * B;                                            // [6][2][B]
  float* etap = edg + 12 * B;                                           // [6 << 6]
  float* btap = etap + (6 << 6);                                        // [3 << 6]
  float* red = reinterpret_cast<float*>(smem);  // [2B][2] once the ring is idle

  const int item = xcd_swizzle(blockIdx.x, gridDim.x);
  const int u = item / a.R, r = item % a.R;
  const long tb = (long)r * a.span;
  const long te = min(tb + (long)a.span, (long)a.L);
  const long L = a.L, nJ = a.nJ;
  const long nb0 = tb >> 6, jend = te >> 6;  // coefficients of this range
  // it owns some of the unit's last three coefficients (symmetric extension)
  const bool sym_end = !periodic && jend > nJ - 3;
  const int nch = (int)((te - tb + CR - 1) / CR);
  // chunks through two blocks past the range (not past the unit with the
  // symmetric extension, whose end coefficients take no rows beyond it)
  const long xe = periodic ? te + CR : min(te + CR, L);
  const int nch_ext = (int)((xe - tb + CR - 1) / CR);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ts = wave & 3, qt = wave >> 2, h = ts & 1;
  const bool loader = qt == 0;
  const int hi = lane >> 5, col = lane & 31;
  const int q = 32 * qt + col;
  const bool live = 32 * qt < B;

  const bf16_t* qrow = reinterpret_cast<const bf16_t*>(a.Q) + ((long)u * B + min(q, B - 1)) * D;
  u32x4 qreg[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) qreg[s] = *reinterpret_cast<const u32x4*>(qrow + 16 * s + 8 * hi);
  for (int i = threadIdx.x; i < (6 << 6); i += kTokBlock) etap[i] = tp.edge[i];
  for (int i = threadIdx.x; i < (3 << 6); i += kTokBlock) btap[i] = tp.band[i];
#pragma unroll
  for (int s = 0; s < KS; ++s) asm volatile("" ::"v"(qreg[s]));
  // the lane's 16 tokens sit at offsets 32 h + 8 g + 4 hi + i (g, i < 4) of
  // their block: taps k of group g are one 16-byte LDS read
  const float* lane_taps = btap + 32 * h + 4 * hi;

  // row r of the chunk at c0: token c0 + r, past the unit wrapped (periodic)
  // or the last row (symmetric: those rows feed no kept coefficient)
  struct Rows {
    const bf16_t* Kunit;
    long c0, L;
    int periodic;
    __device__ __forceinline__ const bf16_t* operator()(int r) const {
      const long p = c0 + r;
      return Kunit + (p < L ? p : (periodic ? p - L : L - 1)) * D;
    }
  } rows{reinterpret_cast<const bf16_t*>(a.K) + (long)u * a.Ls * D, tb, L, periodic};
  const uint32_t ring_lds = lds_offset(ring);
  const int nbuf = a.nbuf;
  if (loader) {
    for (int k = 0; k < nch_ext && k < nbuf - 1; ++k) {
      rows.c0 = tb + (long)k * CR;
      issue_chunk<CR, G, NIW, true>(ring_lds + (uint32_t)(k * CHB), rows);
    }
  }
  const float c2 = a.scale * kLog2e;
  float* out = a.blocks + (long)u * nJ * 2 * B;  // [nJ][2][B]
  // waves 4..7: thread (ci, cq) completes coefficient 2 c + ci of chunk c
  // (held: lane (ci, cq) of wave 4 + c mod 4)
  const int t2 = HOLD ? (wave >= NIW ? lane : -1) : threadIdx.x - NIW * 64;
  const int ci = t2 / B, cq = t2 - ci * B;
  const bool comb = t2 >= 0 && t2 < 2 * B;
  float cm = -INFINITY, cz = 0.f;  // running max / sum of exp of the coarse logits
  f32x32 hl, he;                   // held coarse logits and log-sum-exps (HOLD)
  auto combine = [&](int c) {
    const long n = nb0 + 2L * c + ci;
    if (n >= jend) return;
    float s;
    if (sym_end && n >= nJ - 3) {
      const int m = (int)(nJ - 1 - n);
      const float* ep = edg + (m * (m + 1)) * B + cq;  // (m (m + 1) / 2) * 2 B
      s = 0.f;
      for (int k = 0; k <= m; ++k) s += ep[2 * k * B] + ep[(2 * k + 1) * B];
    } else {
      // slots of chunks c and c + 1: [4 slices][3 partials][B]
      const float* p0 = part + (c % 3) * 12 * B + cq;
      const float* p1 = part + ((c + 1) % 3) * 12 * B + cq;
      const float* pb = ci == 0 ? p0 + 6 * B : p1;  // block n + 1: slices 2, 3 of c or 0, 1 of c + 1
      s = p0[(6 * ci) * B] + p0[(6 * ci + 3) * B];
      s += pb[B] + pb[4 * B];
      s += p1[(6 * ci + 2) * B] + p1[(6 * ci + 5) * B];
    }
    const float l = s * a.scale;
    // the block's log-sum-exp from its two slices (raw maxima: positive scale)
    const float* st = sst + ((c % 3) * 8 + 4 * ci) * B + cq;
    const float m0 = st[0], e0 = st[B], m1 = st[2 * B], e1 = st[3 * B];
    const float mx = fmaxf(m0, m1);
    const float e = e0 * __builtin_amdgcn_exp2f((m0 - mx) * c2) + e1 * __builtin_amdgcn_exp2f((m1 - mx) * c2);
    const float lse = fmaf(mx, a.scale, __logf(e));
    if constexpr (HOLD) {
      const int slot = __builtin_amdgcn_readfirstlane(c >> 2);  // c < 128 (host-checked)
      if (slot < 32) {
        hl[slot] = l;
        he[slot] = lse;
      }
    } else {
      float* o = out + n * 2 * B + cq;
      o[0] = l;
      o[B] = lse;
    }
    stat_add(cm, cz, l);
  };

  // one wave's slice of chunk ch: its partials and statistics into LDS
  auto slice_step = [&](int ch) {
    const unsigned char* buf = ring + (ch % nbuf) * CHB;
    const int row = 32 * ts + col;
    f32x16 acc = {};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const u32x4 ka = *reinterpret_cast<const u32x4*>(buf + granule_offset<G>(row, 2 * s + hi));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, ka),
                                                    __builtin_bit_cast(bf16x8, qreg[s]), acc, 0, 0, 0);
    }
    float mx = acc[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) mx = fmaxf(mx, acc[v]);
    mx = max_xor32(mx);
    const float off = -mx * c2;
    float e = 0.f, p0 = 0.f, p1 = 0.f, p2 = 0.f;
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const f32x4 t0 = *reinterpret_cast<const f32x4*>(lane_taps + 8 * g4);
      const f32x4 t1 = *reinterpret_cast<const f32x4*>(lane_taps + 64 + 8 * g4);
      const f32x4 t2 = *reinterpret_cast<const f32x4*>(lane_taps + 128 + 8 * g4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float x = acc[4 * g4 + i];
        e += __builtin_amdgcn_exp2f(fmaf(x, c2, off));
        p0 = fmaf(t0[i], x, p0);
        p1 = fmaf(t1[i], x, p1);
        p2 = fmaf(t2[i], x, p2);
      }
    }
    e = add_xor32(e);
    p0 = add_xor32(p0);
    p1 = add_xor32(p1);
    p2 = add_xor32(p2);
    const int slot = ch % 3;
    if (hi == 0 && q < B) {
      float* pp = part + ((slot * 4 + ts) * 3) * B + q;
      pp[0] = p0;
      pp[B] = p1;
      pp[2 * B] = p2;
      float* sp = sst + ((slot * 4 + ts) * 2) * B + q;
      sp[0] = mx;
      sp[B] = e;
    }
    if (sym_end) {
      // end-filter partials of the unit's last three blocks
      const long cg = (tb + (long)ch * CR + 32 * ts) >> 6;
      if (cg >= nJ - 3 && cg < nJ) {
#pragma unroll 1
        for (int m = 0; m < 3; ++m) {
          const int k = (int)(cg - (nJ - 1 - m));
          if (k < 0 || k > m) continue;  // uniform
          const float* et = etap + 64 * (m * (m + 1) / 2 + k) + 32 * h + 4 * hi;
          float x = 0.f;
#pragma unroll
          for (int g4 = 0; g4 < 4; ++g4) {
            const f32x4 t = *reinterpret_cast<const f32x4*>(et + 8 * g4);
#pragma unroll
            for (int i = 0; i < 4; ++i) x = fmaf(t[i], acc[4 * g4 + i], x);
          }
          x = add_xor32(x);
          if (hi == 0 && q < B) edg[((m * (m + 1) / 2 + k) * 2 + h) * B + q] = x;
        }
      }
    }
  };

  for (int ch = 0; ch < nch_ext + 2; ++ch) {
    if (loader && ch < nch_ext) wait_vmcnt_chunks<IPW>(min(nch_ext - 1 - ch, nbuf - 2));
    lds_barrier();  // chunk ch in the ring; chunk ch - 1's partials in LDS
    if (loader) {
      if (ch + nbuf - 1 < nch_ext) {
        rows.c0 = tb + (long)(ch + nbuf - 1) * CR;
        issue_chunk<CR, G, NIW, true>(ring_lds + (uint32_t)(((ch + nbuf - 1) % nbuf) * CHB), rows);
      }
    }
    if (ch < nch_ext && live) slice_step(ch);
    if (comb && ch >= 2 && (!HOLD || wave == NIW + ((ch - 2) & 3))) combine(ch - 2);
  }

  if constexpr (HOLD) {
    // slot k of wave 4 + w holds coefficient n0 + 8 k (n0 = nb0 + 2 w + ci):
    // the rows of consecutive slots are 16 B floats apart
    if (comb) {
      const long n0 = nb0 + 2 * (wave - NIW) + ci;
      const int nv = (int)max(0L, min(32L, (jend - n0 + 7) / 8));
      float* o = out + n0 * 2 * B + cq;
      const long stride = 16L * B;
#pragma unroll
      for (int k = 0; k < 32; ++k) {
        if (k < nv) {
          o[(long)k * stride] = hl[k];
          o[(long)k * stride + B] = he[k];
        }
      }
    }
  }

  // the range's (max, sum of exp) per query from the combining threads
  __syncthreads();
  constexpr int NCW = HOLD ? 4 : 1;  // waves whose lanes hold partial pairs
  if (comb) {
    const int idx = HOLD ? (wave - NIW) * 2 * B + t2 : t2;
    red[2 * idx] = cm;
    red[2 * idx + 1] = cz;
  }
  __syncthreads();
  float* ws = a.wstats + ((long)u * a.R + r) * 2 * B;
  for (int qq = threadIdx.x; qq < B; qq += kTokBlock) {
    float m_ = red[2 * qq], z_ = red[2 * qq + 1];
    stat_absorb(m_, z_, red[2 * (B + qq)], red[2 * (B + qq) + 1]);
#pragma unroll
    for (int w = 1; w < NCW; ++w) {
      const float* rw = red + 2 * (w * 2 * B);
      stat_absorb(m_, z_, rw[2 * qq], rw[2 * qq + 1]);
      stat_absorb(m_, z_, rw[2 * (B + qq)], rw[2 * (B + qq) + 1]);
    }
    ws[qq] = m_;
    ws[B + qq] = z_;
  }
}

// W (eq. 8) of every coarse block from the token skim's block rows.  The
// coarse softmax normalisers of a unit are its ranges' (max, sum of exp)
// pairs merged; then W_j = sum_q exp(l_qj - M_q) / Z_q.  Each workgroup takes
// one slice of one unit's blocks, so that the whole GPU reads the block rows
// (one workgroup per unit leaves most of it idle); the top-S selection of
// eq. 9 is taken by the workgroups of the scan that follows.
constexpr int kWeightsBlock = 256;

__global__ __launch_bounds__(kWeightsBlock) void block_weights_kernel(BlockWeightsArgs a) {
  __shared__ float row_c[16 * kFastMaxQBlocks];
  // the unit on the XCD whose L2 took its block rows from the token skim
  const int item = xcd_swizzle(blockIdx.x, gridDim.x);
  const int u = item / a.WPU, slice = item % a.WPU;
  const int B = a.B, nJ = a.nJ;
  const int per = (nJ + a.WPU - 1) / a.WPU;
  const int j0 = slice * per, j1 = min(nJ, j0 + per);
  float* W = a.W + (long)u * nJ;
  unit_block_weights<kWeightsBlock>(a.blocks + (long)u * nJ * 2 * B, a.wstats + (long)u * a.R * 2 * B,
                                    a.R, B, j0, j1, row_c, [&](int j, float w) { W[j] = w; });
}

// The selection weights of the H heads of each sequence added up, h in
// order: one thread per output element, the H loads of a thread issued
// together (consecutive threads read consecutive elements of every head).
constexpr int kHeadSumBlock = 256;

__global__ __launch_bounds__(kHeadSumBlock) void head_sum_kernel(HeadSumArgs a) {
  const long i = (long)blockIdx.x * kHeadSumBlock + threadIdx.x;
  if (i >= (long)a.groups * a.n) return;  // no barrier follows
  const long g = i / a.n, j = i - g * a.n;
  const float* src = a.in + g * a.H * a.n + j;
  float s = 0.f;
#pragma unroll 8
  for (int h = 0; h < a.H; ++h) s += src[(long)h * a.n];
  a.out[i] = s;
}

// ------------------------------------------------------------ host side

bool db2_token_path(const wf_params& p) {
  return p.dtype == WF_BF16 && p.wavelet == WF_DB2 && p.levels == 6 &&
         (p.ctx_len >> 6) >= 4 && p.q_len <= 16 * kFastMaxQBlocks && effective_scale(p) > 0.f;
}

bool fast_path(const wf_params& p) {
  // a positive scale keeps the block maximum of the raw products the maximum
  // of the scaled logits; the scan and attention workgroups keep the unit's
  // region ids in LDS for their selections
  return ((p.dtype == WF_BF16 && p.wavelet == WF_HAAR && p.levels >= 3 && p.levels <= 5 &&
           p.q_len <= 16 * kFastMaxQBlocks && effective_scale(p) > 0.f) ||
          db2_token_path(p)) &&
         p.segments <= kSelectLdsSegs;
}

// LDS of the db2 token skim besides its ring: the partial and statistic
// rings, the end-filter partials and taps
static size_t db2_fixed_lds(int B) { return ((size_t)72 * B + (9 << 6)) * sizeof(float); }

template <bool LSE>
static size_t token_batch_bytes_at(int J, int B) {
  switch (J) {
    case 1: return LSE ? 0 : token_batch_bytes<1, false>(B);
    case 2: return LSE ? 0 : token_batch_bytes<2, false>(B);
    case 3: return token_batch_bytes<3, LSE>(B);
    case 4: return token_batch_bytes<4, LSE>(B);
    default: return token_batch_bytes<5, LSE>(B);
  }
}

// Ranges and ring of the token-level skim with blocks of 2^J tokens over Lf
// rows; `gather`: the rows are a gathered sequence of blocks of 2^(J+1)
// tokens, whose ids each range stages in LDS.
static FastPlan plan_token(const wf_params& p, int J, long Lf, bool lse, bool gather) {
  FastPlan f{};
  const long U = (long)p.batch * p.heads;
  const long chunks = (Lf + kScanChunk - 1) / kScanChunk;
  const size_t chb = (size_t)kScanChunk * 2 * p.head_dim;
  constexpr size_t kLdsPerCu = 160 * 1024;
  // Blocks of 32 tokens with their log-sum-exps: one workgroup per CU that
  // holds its results until its keys are read (token_skim_held_kernel),
  // whenever a range of that shape has at most kHeldChunks chunks.
  if (lse && J == 5 && !gather && !db2_token_path(p) && p.q_len <= 16 * kFastMaxQBlocks) {
    const long R = std::min(chunks, std::max(1L, ((long)device_cu_count() + U - 1) / U));
    const long cpr = (chunks + R - 1) / R;
    if (cpr <= kHeldChunks) {
      f.span = (int)(cpr * kScanChunk);
      f.R = (int)((Lf + f.span - 1) / f.span);
      f.par_cap = 0;
      f.nbuf = (int)std::min<size_t>(3, kLdsPerCu / chb);
      // (the ring also takes the end-of-range reduction pairs, 2 KiB)
      f.lds_bytes = std::max<size_t>((size_t)f.nbuf * chb, 8 * 32 * 2 * sizeof(float));
      f.held = true;
      return f;
    }
  }
  // two batch slots of block results (the db2 skim: its partial rings); the
  // wave reduction pairs reuse the ring
  const size_t bb = db2_token_path(p) ? db2_fixed_lds(p.q_len)
                    : 2 * (lse ? token_batch_bytes_at<true>(J, p.q_len)
                               : token_batch_bytes_at<false>(J, p.q_len));
  // Two resident workgroups per CU, each two chunks deep, stream faster than
  // one three deep (the barrier of one overlaps the other's loads); that
  // shape is taken whenever two fit in the CU's LDS.
  const long want0 = std::max(1L, (2L * device_cu_count() + U - 1) / U);
  const long cpr0 = (chunks + std::min(chunks, want0) - 1) / std::min(chunks, want0);
  const size_t ids = gather ? (size_t)(((cpr0 * kScanChunk) >> (J + 1)) + 2) * 4 : 0;
  const size_t fixed = bb + ((ids + 15) & ~(size_t)15);
  const size_t fit2 = kLdsPerCu / 2 > fixed ? (kLdsPerCu / 2 - fixed) / chb : 0;
  // (the db2 skim needs more than 128 registers a lane: one workgroup per CU)
  const int per_cu = fit2 >= 2 && !db2_token_path(p) &&
                     token_skim_waves_per_simd(p.head_dim, J, lse) >= 4 ? 2 : 1;
  const long want = std::max(1L, ((long)per_cu * device_cu_count() + U - 1) / U);
  const long R = std::min(chunks, want);
  const long cpr = (chunks + R - 1) / R;
  f.span = (int)(cpr * kScanChunk);
  f.R = (int)((Lf + f.span - 1) / f.span);
  // the parent ids of one range (at most span / 2^(J+1) + 2 of them)
  f.par_cap = gather ? (int)((f.span >> (J + 1)) + 2) : 0;
  const size_t fixed2 = bb + (((size_t)f.par_cap * 4 + 15) & ~(size_t)15);
  f.nbuf = (int)std::min<size_t>(3, per_cu == 2 ? (kLdsPerCu / 2 - fixed2) / chb
                                                : (kLdsPerCu - fixed2) / chb);
  f.lds_bytes = f.nbuf * chb + fixed2;
  return f;
}

FastPlan plan_fast(const wf_params& p) {
  return plan_token(p, p.levels, filtered_len(p), true, false);
}

bool rec_token_path(const wf_params& p) {
  return p.dtype == WF_BF16 && p.wavelet == WF_HAAR && p.levels >= 1 && p.levels <= 5 &&
         p.q_len <= 16 * kFastMaxQBlocks;
}

FastPlan plan_rec_token(const wf_params& p, int b, long rows, bool gather) {
  return plan_token(p, b, rows, false, gather);
}

template <int D, int J, bool LSE, bool GATHER = false>
static hipError_t token_skim_launch(const TokenSkimArgs& a, size_t lds, hipStream_t s) {
  auto kern = token_skim_kernel<D, J, LSE, GATHER>;
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)(a.U * a.R)), dim3(kTokBlock), lds, s, a);
  return hipGetLastError();
}

template <int D, bool LSE>
static hipError_t token_skim_dispatch(int J, const TokenSkimArgs& a, size_t lds, hipStream_t s) {
  if constexpr (LSE) {
    switch (J) {
      case 3: return token_skim_launch<D, 3, true>(a, lds, s);
      case 4: return token_skim_launch<D, 4, true>(a, lds, s);
      case 5: return token_skim_launch<D, 5, true>(a, lds, s);
      default: return hipErrorInvalidValue;
    }
  } else if (a.parent) {
    switch (J) {
      case 1: return token_skim_launch<D, 1, false, true>(a, lds, s);
      case 2: return token_skim_launch<D, 2, false, true>(a, lds, s);
      case 3: return token_skim_launch<D, 3, false, true>(a, lds, s);
      case 4: return token_skim_launch<D, 4, false, true>(a, lds, s);
      default: return hipErrorInvalidValue;
    }
  } else {
    switch (J) {
      case 1: return token_skim_launch<D, 1, false>(a, lds, s);
      case 2: return token_skim_launch<D, 2, false>(a, lds, s);
      case 3: return token_skim_launch<D, 3, false>(a, lds, s);
      case 4: return token_skim_launch<D, 4, false>(a, lds, s);
      case 5: return token_skim_launch<D, 5, false>(a, lds, s);
      default: return hipErrorInvalidValue;
    }
  }
}

static TokenSkimArgs token_args(const wf_params& p, const FastPlan& f, int J, long rows,
                                long nJ, const void* Q, const void* K, float* out,
                                float* wstats) {
  TokenSkimArgs a{};
  a.K = K;
  a.Q = Q;
  a.blocks = out;
  a.wstats = wstats;
  a.U = p.batch * p.heads;
  a.L = (int)rows;
  a.Ls = p.ctx_len;
  a.B = p.q_len;
  a.nJ = (int)nJ;
  a.R = f.R;
  a.span = f.span;
  a.nbuf = f.nbuf;
  a.scale = effective_scale(p);
  a.norm = (float)std::pow(2.0, -0.5 * J);
  a.parent = nullptr;
  a.npar = 0;
  a.pshift = J + 1;
  a.par_cap = f.par_cap;
  return a;
}

template <int D, bool HOLD>
static hipError_t token_db2_launch(const TokenSkimArgs& a, const Db2TokenTaps& t, int periodic,
                                   size_t lds, hipStream_t s) {
  auto kern = token_db2_kernel<D, HOLD>;
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)(a.U * a.R)), dim3(kTokBlock), lds, s, a, t, periodic);
  return hipGetLastError();
}

static const Db2TokenTaps& db2_taps6() {
  static Db2TokenTaps t;
  static std::once_flag once;
  std::call_once(once, [] { db2_token_taps(6, &t); });
  return t;
}

hipError_t launch_token_skim(const wf_params& p, const void* Q, const void* K, float* blocks,
                             float* wstats, hipStream_t s) {
  if (!fast_path(p)) return hipErrorInvalidValue;
  const FastPlan f = plan_fast(p);
  if (db2_token_path(p)) {
    const TokenSkimArgs a = token_args(p, f, 6, filtered_len(p), p.ctx_len >> 6, Q, K, blocks,
                                       wstats);
    const int periodic = p.boundary == WF_EXT_PERIODIC ? 1 : 0;
    // block rows held in registers: at most 32 query rows, 128 chunks a range
    const bool hold = p.q_len <= 32 && f.span / kScanChunk <= 128;
    if (hold)
      return p.head_dim == 128
                 ? token_db2_launch<128, true>(a, db2_taps6(), periodic, f.lds_bytes, s)
                 : token_db2_launch<64, true>(a, db2_taps6(), periodic, f.lds_bytes, s);
    return p.head_dim == 128 ? token_db2_launch<128, false>(a, db2_taps6(), periodic, f.lds_bytes, s)
                             : token_db2_launch<64, false>(a, db2_taps6(), periodic, f.lds_bytes, s);
  }
  const TokenSkimArgs a = token_args(p, f, p.levels, filtered_len(p), p.ctx_len >> p.levels, Q,
                                     K, blocks, wstats);
  if (f.held) {
    auto kern = p.head_dim == 128 ? token_skim_held_kernel<128> : token_skim_held_kernel<64>;
    if (f.lds_bytes > 65536) {
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                         hipFuncAttributeMaxDynamicSharedMemorySize,
                                         (int)f.lds_bytes);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, dim3((unsigned)(a.U * a.R)), dim3(kTokBlock), f.lds_bytes, s, a);
    return hipGetLastError();
  }
  return p.head_dim == 128 ? token_skim_dispatch<128, true>(p.levels, a, f.lds_bytes, s)
                           : token_skim_dispatch<64, true>(p.levels, a, f.lds_bytes, s);
}

hipError_t launch_rec_token_skim(const wf_params& p, int b, long n, const int32_t* parent,
                                 int npar, const void* Q, const void* K, float* logits,
                                 float* stats, hipStream_t s) {
  if (!rec_token_path(p) || b < 1 || b > 5) return hipErrorInvalidValue;
  // rows: the filtered keys at the first scale, else the gathered kept blocks
  const long rows = parent ? (long)npar << (b + 1) : filtered_len(p);
  const FastPlan f = plan_rec_token(p, b, rows, parent != nullptr);
  TokenSkimArgs a = token_args(p, f, b, rows, n, Q, K, logits, stats);
  a.parent = parent;
  a.npar = npar;
  return p.head_dim == 128 ? token_skim_dispatch<128, false>(b, a, f.lds_bytes, s)
                           : token_skim_dispatch<64, false>(b, a, f.lds_bytes, s);
}

int weights_slices(const wf_params& p) {
  const long U = (long)p.batch * p.heads;
  const long nJ = (long)p.ctx_len >> p.levels;
  // about four workgroups per CU, at least 16 blocks each
  const long want = (4L * device_cu_count() + U - 1) / U;
  return (int)std::max(1L, std::min(want, (nJ + 15) / 16));
}

hipError_t launch_block_weights(const wf_params& p, const float* blocks, const float* wstats,
                                float* W, hipStream_t s) {
  if (!fast_path(p)) return hipErrorInvalidValue;
  BlockWeightsArgs a;
  a.blocks = blocks;
  a.wstats = wstats;
  a.W = W;
  a.U = p.batch * p.heads;
  a.B = p.q_len;
  a.nJ = p.ctx_len >> p.levels;
  a.R = plan_fast(p).R;
  a.WPU = weights_slices(p);
  hipLaunchKernelGGL(block_weights_kernel, dim3((unsigned)(a.U * a.WPU)), dim3(kWeightsBlock), 0,
                     s, a);
  return hipGetLastError();
}

hipError_t launch_head_sum(const float* in, float* out, long n, int H, int groups,
                           hipStream_t s) {
  if (!in || !out || n < 1 || H < 1 || groups < 1) return hipErrorInvalidValue;
  HeadSumArgs a{in, out, n, H, groups};
  const long total = (long)groups * n;
  hipLaunchKernelGGL(head_sum_kernel, dim3((unsigned)((total + kHeadSumBlock - 1) / kHeadSumBlock)),
                     dim3(kHeadSumBlock), 0, s, a);
  return hipGetLastError();
}

hipError_t load_fast_kernels() {
  hipFuncAttributes fa;
  return hipFuncGetAttributes(&fa, reinterpret_cast<const void*>(head_sum_kernel));
}

}  // namespace wf
