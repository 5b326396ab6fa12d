// Scan: the skim's regions mapped to token indices (eq. 10) and scored at
// token resolution with the same perception-weight procedure (eqs. 7-8 over
// the pool only, Section 3.2), then the top-k tokens (eq. 9) -> mu^0.
//
// The pool of a unit is S runs of 2^J consecutive rows.  It is split into
// chunks of kScanChunk pool positions, one workgroup each.  The softmax over
// the pool needs every chunk's row maximum and normaliser before any weight
// can be formed, so the scan runs as two passes over the chunks:
//   pass 1 (stats):   logits of the chunk on MFMA, per-row max and
//                     sum of exp -> workspace;
//   pass 2 (weights): merge the unit's row statistics, recompute the same
//                     logits (bit-identical: same code and operands), and
//                     W'_p = sum_q exp(s_qp - M_q) / Z_q for the chunk.
// A per-unit select kernel then takes the top-k of W' (ties to the lower
// pool position, which is the lower token index because the regions are
// ascending) and emits token indices in ascending order.
#include "wf_device.hpp"
#include "wf_kernels.hpp"
#include "wf_launch.hpp"

namespace wf {

// Pool chunk staging: row r of a chunk starting at pool position p0 is token
// seg[p >> J] 2^J + (p & (2^J - 1)) with p = p0 + r; rows past the end are
// zero.
template <typename T, int D>
struct PoolRows {
  const T* Kunit;
  const int32_t* seg;
  long p0, last;  // last: the unit's last row (region ids are clamped to it)
  int np, J, mask;
  __device__ __forceinline__ const T* operator()(int r) const {
    if (r >= np) return nullptr;
    const long p = p0 + r;
    const long tok = ((long)seg[p >> J] << J) | (p & mask);
    return Kunit + min(max(tok, 0L), last) * D;
  }
};

template <int WEIGHTS, typename T, int D>
__global__ __launch_bounds__(kBlock) void scan_chunk_kernel(ScanArgs a) {
  using Stager = RowStager<T, D, kScanChunk, kBlock>;
  constexpr int STRIDE = Stager::STRIDE;
  constexpr int NW = kBlock / kWave;
  constexpr int TB = kScanChunk / 16;       // token blocks per chunk
  constexpr int TBW = TB / NW;              // token blocks per wave
  extern __shared__ __align__(16) unsigned char smem[];
  T* Qs = reinterpret_cast<T*>(smem);                       // [B][STRIDE]
  T* Ks = Qs + (size_t)a.B * STRIDE;                         // [chunk][STRIDE]
  float* red = reinterpret_cast<float*>(Ks + kScanChunk * STRIDE);
  const int nqb = (a.B + 15) / 16;
  // stats pass:   part [nqb][NW][16][2] per chunk, run_m [B], run_z [B]
  // weights pass: row_max [B], row_inv [B]
  float* part = red;
  float* run_m = red + nqb * NW * 32;
  float* run_z = run_m + a.B;

  const int item = xcd_swizzle(blockIdx.x, gridDim.x);
  const int u = item / a.C, c = item % a.C;
  const long pb = (long)c * a.span;
  const long pe = min(pb + (long)a.span, (long)a.P);
  const int nchunks = (int)((pe - pb + kScanChunk - 1) / kScanChunk);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, col = lane & 15;
  const T* Qunit = reinterpret_cast<const T*>(a.Q) + (long)u * a.B * D;

  PoolRows<T, D> src;
  src.Kunit = reinterpret_cast<const T*>(a.K) + (long)u * a.Ls * D;
  src.seg = a.seg + (long)(u / a.share) * a.S;
  src.J = a.J;
  src.mask = (1 << a.J) - 1;
  src.last = a.Ls - 1;
  src.p0 = pb;
  src.np = (int)min((long)kScanChunk, pe - pb);
  Stager st;
  st.load(src);

  stage_rows_any<T, D, kBlock>(Qs, a.B, [&](int r) { return Qunit + (long)r * D; });
  if constexpr (WEIGHTS) {
    float* row_max = red;
    float* row_inv = red + a.B;
    const float* stt = a.stats + (long)u * a.Cs * 2 * a.B;
    for (int q = threadIdx.x; q < a.B; q += kBlock) {
      float mx = -INFINITY;
      for (int k = 0; k < a.Cs; ++k) mx = fmaxf(mx, stt[(long)k * 2 * a.B + q]);
      float z = 0.f;
      for (int k = 0; k < a.Cs; ++k) {
        const float mk = stt[(long)k * 2 * a.B + q];
        if (mk > -INFINITY) z += stt[(long)k * 2 * a.B + a.B + q] * __expf(mk - mx);
      }
      row_max[q] = mx;
      row_inv[q] = 1.f / z;
    }
  } else {
    for (int q = threadIdx.x; q < a.B; q += kBlock) {
      run_m[q] = -INFINITY;
      run_z[q] = 0.f;
    }
  }

  for (int ch = 0; ch < nchunks; ++ch) {
    const long p0 = pb + (long)ch * kScanChunk;
    const int np = (int)min((long)kScanChunk, pe - p0);
    __syncthreads();  // the previous chunk's readers are done with Ks
    st.store(Ks);
    __syncthreads();
    if (ch + 1 < nchunks) {
      src.p0 = p0 + kScanChunk;
      src.np = (int)min((long)kScanChunk, pe - src.p0);
      st.load(src);
    }
    float wacc[TBW];
#pragma unroll
    for (int k = 0; k < TBW; ++k) wacc[k] = 0.f;
    for (int qb = 0; qb < nqb; ++qb) {
      const T* arow = Qs + min(qb * 16 + col, a.B - 1) * STRIDE;
      f32x4 sacc[TBW];
#pragma unroll
      for (int k = 0; k < TBW; ++k) {
        const int tb = wave * TBW + k;
        sacc[k] = tile_dot<T, D>(arow, Ks + (tb * 16 + col) * STRIDE,
                                 f32x4{0.f, 0.f, 0.f, 0.f});
      }
      // lane holds logit[q = 16 qb + 4 g + i][p = p0 + 16 tb + col]
      if constexpr (!WEIGHTS) {
        float* rq = part + (qb * NW + wave) * 32;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float mx = -INFINITY;
#pragma unroll
          for (int k = 0; k < TBW; ++k) {
            const bool ok = (wave * TBW + k) * 16 + col < np;
            const float v = ok ? sacc[k][i] * a.scale : -INFINITY;
            sacc[k][i] = v;
            mx = fmaxf(mx, v);
          }
          mx = wave_max16(mx);
          float z = 0.f;
          if (mx > -INFINITY) {
#pragma unroll
            for (int k = 0; k < TBW; ++k)
              if ((wave * TBW + k) * 16 + col < np) z += __expf(sacc[k][i] - mx);
          }
          z = wave_sum16(z);
          if (col == 0) {
            rq[(4 * g + i) * 2] = mx;
            rq[(4 * g + i) * 2 + 1] = z;
          }
        }
      } else {
        const float* row_max = red;
        const float* row_inv = red + a.B;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int q = qb * 16 + 4 * g + i;
          if (q < a.B) {
            const float mq = row_max[q], iz = row_inv[q];
#pragma unroll
            for (int k = 0; k < TBW; ++k)
              wacc[k] += __expf(sacc[k][i] * a.scale - mq) * iz;
          }
        }
      }
    }
    if constexpr (!WEIGHTS) {
      __syncthreads();
      for (int q = threadIdx.x; q < a.B; q += kBlock) {
        const int qb = q >> 4, r = q & 15;
        float mx = run_m[q];
#pragma unroll
        for (int w = 0; w < NW; ++w) mx = fmaxf(mx, part[((qb * NW + w) * 16 + r) * 2]);
        float z = run_m[q] > -INFINITY ? run_z[q] * __expf(run_m[q] - mx) : 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
          const float mw = part[((qb * NW + w) * 16 + r) * 2];
          if (mw > -INFINITY) z += part[((qb * NW + w) * 16 + r) * 2 + 1] * __expf(mw - mx);
        }
        run_m[q] = mx;
        run_z[q] = z;
      }
    } else {
      // column sums over the 4 lane groups (rows 4g + i)
#pragma unroll
      for (int k = 0; k < TBW; ++k) {
        const float w = add_xor32(add_xor16(wacc[k]));
        const int pl = (wave * TBW + k) * 16 + col;
        if (g == 0 && pl < np) a.wpool[(long)u * a.P + p0 + pl] = w;
      }
    }
  }
  if constexpr (!WEIGHTS) {
    __syncthreads();
    float* stt = a.stats + ((long)u * a.Cs + c) * 2 * a.B;
    for (int q = threadIdx.x; q < a.B; q += kBlock) {
      stt[q] = run_m[q];
      stt[a.B + q] = run_z[q];
    }
  }
}

// bf16 pool rows through an LDS ring filled by direct global->LDS loads.
// Row r of the chunk at p0 is pool position min(p0 + r, plast) (rows past
// the range repeat the last valid row and are masked).
template <int D>
struct PoolRowPtr {
  const bf16_t* Kunit;
  const int32_t* segs;  // LDS: region ids from s_lo on
  long p0, plast;
  long last;            // the unit's last row (region ids are clamped to it)
  int J, mask, s_lo;
  __device__ __forceinline__ const bf16_t* operator()(int r) const {
    // row numbers fit in 32 bits (ctx_len <= 2^30)
    const int p = (int)min(p0 + r, plast);
    const int t = (segs[(p >> J) - s_lo] << J) | (p & mask);
    return Kunit + (long)min(max(t, 0), (int)last) * D;
  }
};

// The pool rows of one chunk into a ring slot, as issue_chunk, but every
// row's region id is read from LDS before the first load is issued: an LDS
// read between two of the asm loads waits out its own latency each time.
template <int CR, int G, int NW, bool STREAM, int D>
__device__ __forceinline__ void issue_pool_chunk(uint32_t lds_base, const PoolRowPtr<D>& rowptr) {
  constexpr int RPI = 64 / G;
  constexpr int IPW = CR * G / (64 * NW);
  static_assert(IPW * 64 * NW == CR * G, "chunk must fill whole instructions");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned char* g[IPW];
#pragma unroll
  for (int i = 0; i < IPW; ++i) {
    const int r = (wave * IPW + i) * RPI + lane / G;
    const int k = (lane % G) ^ granule_swz<G>(r);
    g[i] = reinterpret_cast<const unsigned char*>(rowptr(r)) + 16 * k;
  }
#pragma unroll
  for (int i = 0; i < IPW; ++i)
    async_load16<STREAM>(g[i], __builtin_amdgcn_readfirstlane(lds_base + 1024u * (wave * IPW + i)));
}

// 8 waves: two per SIMD, so that one wave's MFMA, exp and LDS latencies
// overlap the other's work (with one wave per SIMD the ring kernel ran at
// well under the gather rate of its memory pattern).
constexpr int kPoolBlock = 512;
constexpr int kPoolWaves = kPoolBlock / kWave;

// SEL (at most 64 query rows): the workgroup first takes the unit's top-S
// regions from W (eq. 9) itself, then queues its first pool chunks.  In the
// weights pass of the token-level path it forms the pool normalisers from
// the selected blocks' log-sum-exps while they load; in the statistics pass
// (the step from cached coefficients) the selection is all it adds, and the
// weights pass that follows reads the region ids the unit's first range
// wrote.
template <int WEIGHTS, int D, bool SEL = false>
__global__ __launch_bounds__(kPoolBlock) void scan_ring_kernel(ScanArgs a) {
  constexpr int NW = kPoolWaves;
  constexpr int CR = kScanChunk;
  constexpr int G = D / 8;             // 16-byte granules per row
  constexpr int CHB = CR * 2 * D;      // bytes per chunk buffer
  constexpr int IPW = CR * G / (64 * NW);
  constexpr int QSTR = D + 8;
  constexpr int TBW = CR / 16 / NW;    // token blocks per wave
  static_assert(TBW >= 1 && TBW * 16 * NW == CR, "whole 16-row blocks per wave");
  constexpr int QPG = 4;               // query blocks held in registers
  constexpr int S32 = D / 32;
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* ring = smem;                                            // [nbuf][CHB]
  bf16_t* Qs = reinterpret_cast<bf16_t*>(smem + (size_t)a.nbuf * CHB);  // [B][QSTR]
  int32_t* segs = reinterpret_cast<int32_t*>(Qs + (size_t)a.B * QSTR);  // [seg_cap]
  float* red = reinterpret_cast<float*>(segs + a.seg_cap);
  const int nqb = (a.B + 15) / 16;
  float* part = red;                   // [nqb][NW][16][2]
  float* lse2 = red + nqb * NW * 32;   // weights: log2 of the pool's sum of exp, per query
  float* wsum = lse2 + a.B;            // weights: W' of the range

  const int item = xcd_swizzle(blockIdx.x, gridDim.x);
  const int u = item / a.C, c = item % a.C;
  const long pb = (long)c * a.span;
  const long pe = min(pb + (long)a.span, (long)a.P);
  const int nch = (int)((pe - pb + CR - 1) / CR);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, col = lane & 15;

  // SEL (at most 64 query rows): the query rows are loaded into registers
  // first and written to LDS after the selection, by when they have landed
  const bf16_t* Qunit = reinterpret_cast<const bf16_t*>(a.Q) + (long)u * a.B * D;
  constexpr int QVR = D / 8;                                  // 16-byte vectors per row
  constexpr int QV = (64 * QVR + kPoolBlock - 1) / kPoolBlock;  // vectors per thread
  const int qtotal = a.B * QVR;
  u32x4 qpre[QV];
  if constexpr (SEL) {
#pragma unroll
    for (int i = 0; i < QV; ++i) {
      const int v = min(i * kPoolBlock + (int)threadIdx.x, qtotal - 1);
      qpre[i] = *reinterpret_cast<const u32x4*>(Qunit + (long)(v / QVR) * D + (v % QVR) * 8);
    }
  }

  // region ids of this range: the span's own, or with SEL all S of the unit
  const int s_lo = SEL ? 0 : (int)(pb >> a.J);
  const uint32_t ring_lds = lds_offset(ring);
  const int nbuf = a.nbuf;
  PoolRowPtr<D> rp;
  rp.Kunit = reinterpret_cast<const bf16_t*>(a.K) + (long)u * a.Ls * D;
  rp.segs = segs;
  rp.plast = pe - 1;
  rp.last = a.Ls - 1;
  rp.J = a.J;
  rp.mask = (1 << a.J) - 1;
  rp.s_lo = s_lo;
  if constexpr (SEL) {
    // top-S of W: the selection's histograms in the last ring slot, and
    // past the register select's reach W in the slots before it when it
    // fits (the ring is free until the first chunks are queued below)
    unsigned char* spare = ring + (size_t)(nbuf - 1) * CHB;
    auto& sh = *reinterpret_cast<SelectShared<kPoolBlock>*>(spare);
    float* Wl = reinterpret_cast<float*>(ring);
    const int sel = u / a.share;  // the unit's selection
    const float* Wg = a.W + (long)sel * a.nJ;
    int32_t* seg_out = c == 0 && u % a.share == 0 ? a.seg_out + (long)sel * a.S : nullptr;
    auto emit = [&](uint32_t pos, int j) {
      segs[pos] = j;
      if (seg_out) seg_out[pos] = j;
    };
    constexpr int EPT = 16;  // weights per thread held in registers
    if (a.nJ <= EPT * kPoolBlock) {
      block_select_topk_regs<kPoolBlock, EPT>(Wg, a.nJ, a.S, emit, sh);
    } else {
      if (a.w_in_lds) {
        for (int i = threadIdx.x; i < a.nJ; i += kPoolBlock) Wl[i] = Wg[i];
        __syncthreads();
        block_select_topk<kPoolBlock>(Wl, a.nJ, a.S, emit, sh);
      } else {
        block_select_topk<kPoolBlock>(Wg, a.nJ, a.S, emit, sh);
      }
    }
    __syncthreads();
    // the first chunks load while the normalisers are formed (the weights
    // pass reads the pool for the last time: streaming loads)
    for (int k = 0; k < nch && k < nbuf - 1; ++k) {
      rp.p0 = pb + (long)k * CR;
      issue_pool_chunk<CR, G, NW, (bool)WEIGHTS>(ring_lds + (uint32_t)(k * CHB), rp);
    }
    if constexpr (WEIGHTS) {
      // pool normalisers (M_q, Z_q) over the pool's tokens, from the selected
      // blocks' log-sum-exps: thread (part, q) folds blocks part, part +
      // parts, ...; the parts' pairs meet in the spare slot
      const int B = a.B;
      const int parts = min(kPoolBlock / B, 16);
      float* pm = reinterpret_cast<float*>(spare);  // [parts][B + 1]
      float* pz = pm + 16 * (B + 1);
      {
        const int q = threadIdx.x % B, part = threadIdx.x / B;
        const float* lse = a.blocks + (long)u * a.nJ * 2 * B + B;  // block j: at (2 j + 1) B
        if (part < parts) {
          float mx = -INFINITY, z = 0.f;
          constexpr int BATCH = 8;  // loads in flight together
          for (int s0 = part; s0 < a.S; s0 += BATCH * parts) {
            float v[BATCH];
  #pragma unroll
            for (int k = 0; k < BATCH; ++k) {
              const int s_ = s0 + parts * k;
              v[k] = s_ < a.S ? lse[(long)segs[s_] * 2 * B + q] : -INFINITY;
            }
  #pragma unroll
            for (int k = 0; k < BATCH; ++k) stat_absorb(mx, z, v[k], 1.f);
          }
          pm[part * (B + 1) + q] = mx;
          pz[part * (B + 1) + q] = z;
        }
      }
      __syncthreads();
      for (int q = threadIdx.x; q < B; q += kPoolBlock) {
        float mx = -INFINITY, z = 0.f;
        for (int k = 0; k < parts; ++k) stat_absorb(mx, z, pm[k * (B + 1) + q], pz[k * (B + 1) + q]);
        // exp(s - M) / Z = 2^(s log2(e) - (M log2(e) + log2(Z)))
        lse2[q] = fmaf(mx, kLog2e, __log2f(z));
      }
    }
  } else {
    const int ns = (int)((pe - 1) >> a.J) - s_lo + 1;
    const int32_t* useg = a.seg + (long)(u / a.share) * a.S;  // the unit's selection
    for (int i = threadIdx.x; i < ns; i += kPoolBlock) segs[i] = useg[s_lo + i];
  }
  if constexpr (SEL) {
#pragma unroll
    for (int i = 0; i < QV; ++i) {
      const int v = i * kPoolBlock + (int)threadIdx.x;
      if (v < qtotal) *reinterpret_cast<u32x4*>(Qs + (v / QVR) * QSTR + (v % QVR) * 8) = qpre[i];
    }
  } else {
    stage_rows_any<bf16_t, D, kPoolBlock>(Qs, a.B, [&](int r) { return Qunit + (long)r * D; });
  }
  if constexpr (WEIGHTS && !SEL) {
    const float* stt = a.stats + (long)u * a.Cs * 2 * a.B;
    for (int q = threadIdx.x; q < a.B; q += kPoolBlock) {
      float mx = -INFINITY, z = 0.f;
      constexpr int SB = 8;  // slices whose loads are in flight together
      for (int k0 = 0; k0 < a.Cs; k0 += SB) {
        float mk[SB], zk[SB];
#pragma unroll
        for (int k = 0; k < SB; ++k) {
          const bool ok = k0 + k < a.Cs;
          mk[k] = ok ? stt[(long)(k0 + k) * 2 * a.B + q] : -INFINITY;
          zk[k] = ok ? stt[(long)(k0 + k) * 2 * a.B + a.B + q] : 0.f;
        }
#pragma unroll
        for (int k = 0; k < SB; ++k) stat_absorb(mx, z, mk[k], zk[k]);
      }
      // exp(s - M) / Z = 2^(s log2(e) - (M log2(e) + log2(Z)))
      lse2[q] = fmaf(mx, kLog2e, __log2f(z));
    }
  }
  __syncthreads();  // every regular load above has been consumed

  const float s2 = a.scale * kLog2e;
  // LDS byte offsets of the lane's key operands: the same rows of every chunk
  int boff[TBW][S32];
#pragma unroll
  for (int k = 0; k < TBW; ++k)
#pragma unroll
    for (int s = 0; s < S32; ++s) boff[k][s] = granule_offset<G>((wave * TBW + k) * 16 + col, 4 * s + g);
  for (int qg = 0; qg < nqb; qg += QPG) {
    // query operands of this group, in registers for the whole range
    u32x4 qreg[QPG][S32];
#pragma unroll
    for (int j = 0; j < QPG; ++j) {
      const bf16_t* arow = Qs + min((qg + j) * 16 + col, a.B - 1) * QSTR;
#pragma unroll
      for (int s = 0; s < S32; ++s)
        qreg[j][s] = *reinterpret_cast<const u32x4*>(arow + 32 * s + 8 * g);
    }
    // weights: the log2-domain normalisers of the lane's query rows (rows
    // past B contribute 2^-inf = 0)
    float c2[QPG][4];
#pragma unroll
    for (int j = 0; j < QPG; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = (qg + j) * 16 + 4 * g + i;
        c2[j][i] = WEIGHTS && q < a.B ? lse2[q] : INFINITY;
      }
    float sm[QPG][4], sz[QPG][4];  // per-lane running row max / sum of exp
#pragma unroll
    for (int j = 0; j < QPG; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sm[j][i] = -INFINITY;
        sz[j][i] = 0.f;
      }
    // ring of nbuf slots, nbuf - 1 chunks in flight ahead of the one consumed.
    // The weights pass reads each pool row for the last time with the
    // streaming (nt) policy: keeping the rows cached measured slower (the
    // attention that follows loads the selected keys with nt as well).
    for (int k = 0; k < nch && k < nbuf - 1 && !(SEL && qg == 0); ++k) {
      rp.p0 = pb + (long)k * CR;
      issue_pool_chunk<CR, G, NW, (bool)WEIGHTS>(ring_lds + (uint32_t)(k * CHB), rp);
    }
    for (int ch = 0; ch < nch; ++ch) {
      const long p0 = pb + (long)ch * CR;
      const int np = (int)min((long)CR, pe - p0);
      wait_vmcnt_chunks<IPW>(min(nch - 1 - ch, nbuf - 2));
      lds_barrier();  // chunk ch visible; everyone is past chunk ch - 1
      if (ch + nbuf - 1 < nch) {
        rp.p0 = pb + (long)(ch + nbuf - 1) * CR;
        issue_pool_chunk<CR, G, NW, (bool)WEIGHTS>(ring_lds + (uint32_t)(((ch + nbuf - 1) % nbuf) * CHB), rp);
      }
      const unsigned char* buf = ring + (ch % nbuf) * CHB;
#pragma unroll
      for (int k = 0; k < TBW; ++k) {
        const int row = (wave * TBW + k) * 16 + col;
        const bool ok = row < np;
        u32x4 bv[S32];
#pragma unroll
        for (int s = 0; s < S32; ++s) bv[s] = *reinterpret_cast<const u32x4*>(buf + boff[k][s]);
        // the query blocks' products interleaved: independent accumulators
        // (blocks past B use clamped query rows; their results are unused)
        f32x4 acc[QPG];
#pragma unroll
        for (int j = 0; j < QPG; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < S32; ++s)
#pragma unroll
          for (int j = 0; j < QPG; ++j)
            acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, qreg[j][s]), __builtin_bit_cast(bf16x8, bv[s]),
                acc[j], 0, 0, 0);
        float wk = 0.f;
#pragma unroll
        for (int j = 0; j < QPG; ++j) {
          if (qg + j >= nqb) break;
          // lane holds logit[q = 16 (qg + j) + 4 g + i][p = p0 + row]
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if constexpr (!WEIGHTS) {
              const float v = acc[j][i] * a.scale;
              if (ok) {
                if (v > sm[j][i]) {
                  sz[j][i] = sz[j][i] * __expf(sm[j][i] - v) + 1.f;
                  sm[j][i] = v;
                } else {
                  sz[j][i] += __expf(v - sm[j][i]);
                }
              }
            } else {
              wk += __builtin_amdgcn_exp2f(fmaf(acc[j][i], s2, -c2[j][i]));
            }
          }
        }
        if constexpr (WEIGHTS) {
          wk = add_xor32(add_xor16(wk));
          // query groups add up in place: the same lane owns this position
          // in every group
          if (g == 0 && ok) wsum[p0 - pb + row] = (qg == 0 ? 0.f : wsum[p0 - pb + row]) + wk;
        }
      }
    }
    if constexpr (!WEIGHTS) {
      // merge the 16 lanes of each row, then the waves, through LDS
#pragma unroll
      for (int j = 0; j < QPG; ++j) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          row16_merge<8>(sm[j][i], sz[j][i]);
          row16_merge<4>(sm[j][i], sz[j][i]);
          row16_merge<2>(sm[j][i], sz[j][i]);
          row16_merge<1>(sm[j][i], sz[j][i]);
          if (col == 0 && qg + j < nqb) {
            part[(((qg + j) * NW + wave) * 16 + 4 * g + i) * 2] = sm[j][i];
            part[(((qg + j) * NW + wave) * 16 + 4 * g + i) * 2 + 1] = sz[j][i];
          }
        }
      }
    }
    lds_barrier();  // the ring is idle; `part` / `wsum` complete
  }
  if constexpr (!WEIGHTS) {
    float* stt = a.stats + ((long)u * a.Cs + c) * 2 * a.B;
    for (int q = threadIdx.x; q < a.B; q += kPoolBlock) {
      const int qb = q >> 4, r = q & 15;
      float mx = -INFINITY, z = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w)
        stat_absorb(mx, z, part[((qb * NW + w) * 16 + r) * 2], part[((qb * NW + w) * 16 + r) * 2 + 1]);
      stt[q] = mx;
      stt[a.B + q] = z;
    }
  } else {
    float* dst = a.wpool + (long)u * a.P + pb;
    for (int i = threadIdx.x; i < (int)(pe - pb); i += kPoolBlock) dst[i] = wsum[i];
  }
}

constexpr int kScanSelectBlock = 1024;

__global__ __launch_bounds__(kScanSelectBlock) void scan_select_kernel(
    ScanSelectArgs a, int w_in_lds, int seg_in_lds) {
  __shared__ SelectShared<kScanSelectBlock> sh;
  extern __shared__ float wsh[];
  const int u = blockIdx.x;
  const float* W = a.wpool + (long)u * a.P;
  // the unit's region ids, read by the emits (from LDS when they fit)
  const int32_t* seg = a.seg + (long)u * a.S;
  if (seg_in_lds) {
    int32_t* seg_sh = reinterpret_cast<int32_t*>(wsh + (w_in_lds ? a.P : 0));
    for (int i = threadIdx.x; i < a.S; i += kScanSelectBlock) seg_sh[i] = seg[i];
    seg = seg_sh;
  }
  if (w_in_lds)
    for (int i = threadIdx.x; i < a.P; i += kScanSelectBlock) wsh[i] = W[i];
  __syncthreads();
  const int J = a.J;
  const int mask = (1 << J) - 1;
  int32_t* tok = a.tok + (long)u * a.keff;
  auto emit = [&](uint32_t pos, int p) { tok[pos] = (seg[p >> J] << J) | (p & mask); };
  // one instance per address space of the weights
  if (w_in_lds)
    block_select_topk<kScanSelectBlock>(wsh, a.P, a.keff, emit, sh);
  else
    block_select_topk<kScanSelectBlock>(W, a.P, a.keff, emit, sh);
}

// ------------------------------------------------------------ host side

// LDS a workgroup may use (gfx950: 160 KiB per CU), with a little margin.
constexpr size_t kLdsBudget = 160 * 1024 - 1024;

ScanPlan plan_scan(const wf_params& p, bool select) {
  ScanPlan s{};
  const long P = (long)p.segments << p.levels;
  const long U = (long)p.batch * p.heads;
  const long chunks = (P + kScanChunk - 1) / kScanChunk;
  const int nqb = (p.q_len + 15) / 16;
  if (p.dtype == WF_BF16) {
    // one workgroup per CU, each streaming a long range through the ring
    const long want = std::max(1L, (long)(device_cu_count() + U - 1) / U);
    long C = std::min(chunks, want);
    long cpw = (chunks + C - 1) / C;
    cpw = std::min(cpw, 32L);  // at most 4096 positions per workgroup
    s.span = (int)(cpw * kScanChunk);
    s.chunks = (int)((P + s.span - 1) / s.span);
    // region ids in LDS: the span's, or all S when the scan selects them
    s.seg_cap = select ? p.segments : (s.span >> p.levels) + 2;
    const size_t chb = (size_t)kScanChunk * 2 * p.head_dim;
    // wave partials, the per-query normalisers, then W' of the range
    const size_t red_ring =
        ((size_t)nqb * kPoolWaves * 16 * 2 + (size_t)p.q_len + (size_t)s.span) * sizeof(float);
    const size_t other = (size_t)p.q_len * (p.head_dim + 8) * 2 + (size_t)s.seg_cap * 4 + red_ring;
    // three slots (two chunks in flight) measured slightly faster than four
    s.nbuf = (int)std::min<size_t>(3, (kLdsBudget - std::min(other, kLdsBudget)) / chb);
    s.lds_bytes = s.nbuf * chb + other;
    if (s.nbuf < 2) s.nbuf = 0;  // rejected by the caller
    return s;
  }
  // fp32: register-staged chunks, about 1024 workgroups of 1..8 chunks
  const long cpw = std::max(1L, std::min(8L, U * chunks / 1024));
  s.span = (int)(cpw * kScanChunk);
  s.chunks = (int)((P + s.span - 1) / s.span);
  const size_t stride = (size_t)p.head_dim * 4 + 16;
  const size_t red_base = ((size_t)nqb * 4 * 16 * 2 + (size_t)2 * p.q_len) * sizeof(float);
  s.lds_bytes = (size_t)(p.q_len + kScanChunk) * stride + red_base;
  return s;
}

template <class Kernel>
static hipError_t launch_with_lds(Kernel kern, dim3 grid, int block, size_t lds, hipStream_t s,
                                  const ScanArgs& a) {
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, grid, dim3(block), lds, s, a);
  return hipGetLastError();
}

template <int WEIGHTS, typename T, int D>
static hipError_t scan_launch(const ScanArgs& a, size_t lds, hipStream_t s) {
  const dim3 grid((unsigned)(a.U * a.C));
  if constexpr (sizeof(T) == 2)
    return launch_with_lds(scan_ring_kernel<WEIGHTS, D>, grid, kPoolBlock, lds, s, a);
  else
    return launch_with_lds(scan_chunk_kernel<WEIGHTS, T, D>, grid, kBlock, lds, s, a);
}

// the scan's arguments when its workgroups take the top-S regions from W
// themselves; false when the shape does not allow it
static bool scan_select_args(const wf_params& p, const void* Q, const void* K, const float* W,
                             int32_t* seg_out, int share, ScanArgs& a, ScanPlan& pl) {
  if (p.dtype != WF_BF16 || p.q_len > 64 || p.segments > kSelectLdsSegs || share < 1 ||
      (p.batch * p.heads) % share != 0)
    return false;
  pl = plan_scan(p, true);
  if (pl.nbuf < 2) return false;
  a = ScanArgs{};
  a.Q = Q;
  a.K = K;
  a.W = W;
  a.share = share;
  a.seg_out = seg_out;
  a.U = p.batch * p.heads;
  a.L = (int)filtered_len(p);
  a.Ls = p.ctx_len;
  a.B = p.q_len;
  a.J = p.levels;
  a.S = p.segments;
  a.P = p.segments << p.levels;
  a.nJ = p.ctx_len >> p.levels;
  a.C = pl.chunks;
  a.span = pl.span;
  a.nbuf = pl.nbuf;
  a.seg_cap = pl.seg_cap;
  a.scale = effective_scale(p);
  // W in the ring slots before the spare one when it fits there
  const size_t chb = (size_t)kScanChunk * 2 * p.head_dim;
  a.w_in_lds = (size_t)a.nJ * sizeof(float) <= (size_t)(pl.nbuf - 1) * chb ? 1 : 0;
  return true;
}

bool scan_can_select(const wf_params& p) {
  ScanArgs a;
  ScanPlan pl;
  return scan_select_args(p, nullptr, nullptr, nullptr, nullptr, 1, a, pl);
}

hipError_t launch_scan_select_weights(const wf_params& p, const void* Q, const void* K,
                                      const float* W, const float* blocks, int32_t* seg_out,
                                      float* wpool, hipStream_t s, int share) {
  ScanArgs a;
  ScanPlan pl;
  if (!scan_select_args(p, Q, K, W, seg_out, share, a, pl)) return hipErrorInvalidValue;
  a.blocks = blocks;
  a.wpool = wpool;
  a.Cs = 1;
  const dim3 grid((unsigned)(a.U * a.C));
  if (p.head_dim == 128)
    return launch_with_lds(scan_ring_kernel<1, 128, true>, grid, kPoolBlock, pl.lds_bytes, s, a);
  return launch_with_lds(scan_ring_kernel<1, 64, true>, grid, kPoolBlock, pl.lds_bytes, s, a);
}

hipError_t launch_scan_select_stats(const wf_params& p, const void* Q, const void* K,
                                    const float* W, int32_t* seg_out, float* stats,
                                    hipStream_t s) {
  ScanArgs a;
  ScanPlan pl;
  if (!scan_select_args(p, Q, K, W, seg_out, 1, a, pl)) return hipErrorInvalidValue;
  a.stats = stats;
  a.Cs = pl.chunks;
  const dim3 grid((unsigned)(a.U * a.C));
  if (p.head_dim == 128)
    return launch_with_lds(scan_ring_kernel<0, 128, true>, grid, kPoolBlock, pl.lds_bytes, s, a);
  return launch_with_lds(scan_ring_kernel<0, 64, true>, grid, kPoolBlock, pl.lds_bytes, s, a);
}

hipError_t launch_scan_chunks(const wf_params& p, int weights, const void* Q,
                              const void* K, const int32_t* seg, float* stats,
                              float* wpool, hipStream_t s, int stat_slices, int share) {
  if (share < 1 || (p.batch * p.heads) % share != 0) return hipErrorInvalidValue;
  const ScanPlan pl = plan_scan(p);
  ScanArgs a;
  a.share = share;
  a.Q = Q;
  a.K = K;
  a.seg = seg;
  a.stats = stats;
  a.wpool = wpool;
  a.U = p.batch * p.heads;
  a.L = (int)filtered_len(p);
  a.Ls = p.ctx_len;
  a.B = p.q_len;
  a.J = p.levels;
  a.S = p.segments;
  a.P = p.segments << p.levels;
  a.C = pl.chunks;
  a.Cs = stat_slices > 0 ? stat_slices : pl.chunks;
  a.span = pl.span;
  a.nbuf = pl.nbuf;
  a.seg_cap = pl.seg_cap;
  a.scale = effective_scale(p);
  const bool bf = p.dtype == WF_BF16, d128 = p.head_dim == 128;
  if (weights) {
    if (bf) return d128 ? scan_launch<1, bf16_t, 128>(a, pl.lds_bytes, s)
                        : scan_launch<1, bf16_t, 64>(a, pl.lds_bytes, s);
    return d128 ? scan_launch<1, float, 128>(a, pl.lds_bytes, s)
                : scan_launch<1, float, 64>(a, pl.lds_bytes, s);
  }
  if (bf) return d128 ? scan_launch<0, bf16_t, 128>(a, pl.lds_bytes, s)
                      : scan_launch<0, bf16_t, 64>(a, pl.lds_bytes, s);
  return d128 ? scan_launch<0, float, 128>(a, pl.lds_bytes, s)
              : scan_launch<0, float, 64>(a, pl.lds_bytes, s);
}

hipError_t launch_scan_select(const wf_params& p, const float* wpool,
                              const int32_t* seg, int32_t* tok,
                              hipStream_t s) {
  ScanSelectArgs a;
  a.wpool = wpool;
  a.seg = seg;
  a.tok = tok;
  a.U = p.batch * p.heads;
  a.J = p.levels;
  a.S = p.segments;
  a.P = p.segments << p.levels;
  a.keff = wf_effective_budget(&p);
  const int in_lds = a.P <= kSelectLdsFloats ? 1 : 0;
  const int seg_in_lds = a.S <= kSelectLdsSegs ? 1 : 0;
  // W' when it fits, then the region ids when they fit
  const size_t lds =
      ((in_lds ? (size_t)a.P : 0) + (seg_in_lds ? (size_t)a.S : 0)) * sizeof(float);
  if (lds > 32768) {  // with the static arrays, past the default 64 KiB
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(scan_select_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(scan_select_kernel, dim3((unsigned)a.U),
                     dim3(kScanSelectBlock), lds, s, a, in_lds, seg_in_lds);
  return hipGetLastError();
}

hipError_t load_scan_kernels() {
  hipFuncAttributes fa;
  return hipFuncGetAttributes(&fa, reinterpret_cast<const void*>(scan_select_kernel));
}

}  // namespace wf
