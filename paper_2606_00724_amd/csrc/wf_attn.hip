// Sparse cache and attention over it (Section 3.2, last paragraph; the
// cached-attention form of eq. 3, bidirectional: no mask).
//
// The cache rows of a unit are split into chunks of kAttnChunk rows, one
// workgroup each (split-KV); each workgroup writes its unnormalised partial
// output with the per-row max and sum of exp, and a combine kernel merges the
// splits.  In the fused path the rows are read in place: row r < k_eff is
// K[tok[r]] / V[tok[r]], the rest are the tail rows K_g / V_g.
//
// bf16: S^T = K Q^T runs on v_mfma_f32_16x16x32_bf16 over 32-row sub-blocks.
// The two 16-row MFMA tiles of a sub-block take rows 8(m/4) + m%4 and
// 8(m/4) + 4 + m%4, so that lane group g ends up holding the scores of rows
// 8g .. 8g+7 for query l%16 -- exactly the A operand of O = P V for the same
// instruction.  V sits transposed in LDS so that its B operand is one 16-byte
// read.  Online softmax (running max / sum per query row) spans the
// sub-blocks.  fp32 uses v_mfma_f32_16x16x4_f32 on 16-row sub-blocks.
#include <type_traits>

#include "wf_device.hpp"
#include "wf_kernels.hpp"
#include "wf_launch.hpp"

namespace wf {

// Absolute cache row rr of unit u: K[tok[rr]] for rr < nsel, then the tail
// rows; contiguous rows when tok is null.  Rows outside [r_lo, r_hi) of the
// current chunk are zero.
template <typename T, int D>
struct CacheRows {
  const T* base;
  const T* tail;
  const int32_t* tok;   // unit's token list or null
  long unit_rows;       // rows per unit in `base` (L, or nrows when contiguous)
  long Lf;              // rows Lf .. Lf + R - 1 of `base` follow the token list
  int u, nsel, G, R;
  long r0;
  int nr;
  __device__ __forceinline__ const T* operator()(int r) const {
    if (r >= nr) return nullptr;
    const long rr = r0 + r;
    if (tok) {
      if (rr < nsel)
        return base + ((long)u * unit_rows + min(max((long)tok[rr], 0L), unit_rows - 1)) * D;
      if (rr < nsel + R) return base + ((long)u * unit_rows + Lf + (rr - nsel)) * D;
      return tail + ((long)u * G + (rr - nsel - R)) * D;
    }
    return base + ((long)u * unit_rows + rr) * D;
  }
};

// bf16 V chunk in token-pair layout: dword [m][c] holds channel c of rows
// 2m (low half) and 2m+1 (high half), so the PV operand of rows 8g .. 8g+7
// is four dword reads.  Thread t stages pairs of 8-channel vectors.
template <int D, int NT>
struct VPairStager {
  static constexpr int VPR = D / 8;                       // vectors per row
  static constexpr int ITEMS = (kAttnChunk / 2) * VPR;    // (pair, vector)
  static constexpr int PER_THREAD = (ITEMS + NT - 1) / NT;
  static constexpr int VPS = D + 4;                       // dwords per pair row
  u32x4 lo[PER_THREAD], hi[PER_THREAD];

  template <class Src>
  __device__ __forceinline__ void load(const Src& src) {
    const bf16_t* pa[PER_THREAD];
    const bf16_t* pb[PER_THREAD];
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int v = i * NT + threadIdx.x;
      const int m = v / VPR;
      pa[i] = v < ITEMS ? src(2 * m) : nullptr;
      pb[i] = v < ITEMS ? src(2 * m + 1) : nullptr;
    }
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int k = (i * NT + threadIdx.x) % VPR;
      lo[i] = pa[i] ? *reinterpret_cast<const u32x4*>(pa[i] + 8 * k) : u32x4{0u, 0u, 0u, 0u};
      hi[i] = pb[i] ? *reinterpret_cast<const u32x4*>(pb[i] + 8 * k) : u32x4{0u, 0u, 0u, 0u};
    }
  }

  __device__ __forceinline__ void store(uint32_t* dst) const {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int v = i * NT + threadIdx.x;
      if (v < ITEMS) {
        const int m = v / VPR, k = v % VPR;
        u32x4 w0, w1;
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          w0[2 * e] = (lo[i][e] & 0xffffu) | (hi[i][e] << 16);
          w0[2 * e + 1] = (lo[i][e] >> 16) | (hi[i][e] & 0xffff0000u);
          w1[2 * e] = (lo[i][e + 2] & 0xffffu) | (hi[i][e + 2] << 16);
          w1[2 * e + 1] = (lo[i][e + 2] >> 16) | (hi[i][e + 2] & 0xffff0000u);
        }
        uint32_t* row = dst + m * VPS + 8 * k;
        *reinterpret_cast<u32x4*>(row) = w0;
        *reinterpret_cast<u32x4*>(row + 4) = w1;
      }
    }
  }
};

template <typename T, int D>
__global__ __launch_bounds__(kBlock) void attn_kernel(AttnArgs a) {
  constexpr int NW = kBlock / kWave;
  constexpr bool BF = sizeof(T) == 2;
  using KStager = RowStager<T, D, kAttnChunk, kBlock>;
  constexpr int KSTR = KStager::STRIDE;
  using VStage = typename std::conditional<BF, VPairStager<D, kBlock>,
                                           RowStager<T, D, kAttnChunk, kBlock>>::type;
  // fp32 V is row-major with stride D + 4 floats; bf16 V is the pair layout
  constexpr int VPS = D + 4;
  extern __shared__ __align__(16) unsigned char smem[];
  T* Ks = reinterpret_cast<T*>(smem);
  uint32_t* Vl = reinterpret_cast<uint32_t*>(Ks + kAttnChunk * KSTR);

  const int item = xcd_swizzle(blockIdx.x, gridDim.x);
  const int u = item / a.NS, sp = item % a.NS;
  const long rb0 = (long)sp * a.rps;
  const long re0 = min(rb0 + (long)a.rps, (long)a.nrows);
  const int nchunks = (int)((re0 - rb0 + kAttnChunk - 1) / kAttnChunk);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, col = lane & 15;

  CacheRows<T, D> ksrc, vsrc;
  ksrc.base = reinterpret_cast<const T*>(a.K);
  vsrc.base = reinterpret_cast<const T*>(a.V);
  ksrc.tail = reinterpret_cast<const T*>(a.Kg);
  vsrc.tail = reinterpret_cast<const T*>(a.Vg);
  ksrc.tok = vsrc.tok = a.tok ? a.tok + (long)(u / a.share) * a.nsel : nullptr;
  ksrc.unit_rows = vsrc.unit_rows = a.tok ? (long)a.L : (long)a.nrows;
  ksrc.u = vsrc.u = u;
  ksrc.nsel = vsrc.nsel = a.nsel;
  ksrc.G = vsrc.G = a.G;
  ksrc.R = vsrc.R = a.R;
  ksrc.Lf = vsrc.Lf = a.Lf;

  const int nqb = (a.B + 15) / 16;
  const int tsplit = nqb == 1 ? 4 : (nqb == 2 ? 2 : 1);
  const int qpg = NW / tsplit;                 // query blocks per group
  const int ngroups = (nqb + qpg - 1) / qpg;
  const int part = wave % tsplit;
  const int R = kAttnChunk / tsplit;           // chunk rows per wave
  const T* Qunit = reinterpret_cast<const T*>(a.Q) + (long)u * a.B * D;
  float* po_base = a.part + ((long)u * a.NS + sp) * a.B * D;
  float* ps_base = a.pstat + ((long)u * a.NS + sp) * 2 * a.B;

  KStager kst;
  VStage vst;
  for (int grp = 0; grp < ngroups; ++grp) {
    const int qb = grp * qpg + wave / tsplit;
    const bool active = qb < nqb;
    const T* qrow = Qunit + (long)min(qb * 16 + col, a.B - 1) * D;
    f32x4 O[D / 16];
#pragma unroll
    for (int cb = 0; cb < D / 16; ++cb) O[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;
    u32x4 qreg[BF ? D / 32 : 1];
    if constexpr (BF) {
#pragma unroll
      for (int s = 0; s < D / 32; ++s)
        qreg[s] = *reinterpret_cast<const u32x4*>(qrow + 32 * s + 8 * g);
    }
    ksrc.r0 = vsrc.r0 = rb0;
    ksrc.nr = vsrc.nr = (int)min((long)kAttnChunk, re0 - rb0);
    kst.load(ksrc);
    vst.load(vsrc);
    for (int ch = 0; ch < nchunks; ++ch) {
      const int nr = (int)min((long)kAttnChunk, re0 - (rb0 + (long)ch * kAttnChunk));
      __syncthreads();  // previous chunk (or group) done with the LDS
      kst.store(Ks);
      if constexpr (BF) vst.store(Vl);
      else vst.store(reinterpret_cast<T*>(Vl));
      __syncthreads();
      if (ch + 1 < nchunks) {
        ksrc.r0 = vsrc.r0 = rb0 + (long)(ch + 1) * kAttnChunk;
        ksrc.nr = vsrc.nr = (int)min((long)kAttnChunk, re0 - ksrc.r0);
        kst.load(ksrc);
        vst.load(vsrc);
      }
      if (!active) continue;
      const int rb = part * R;
      const int re = min(rb + R, nr);
      if constexpr (BF) {
        for (int sb = rb; sb < re; sb += 32) {
          const int rx = sb + 8 * (col >> 2) + (col & 3);
          f32x4 ax = {0.f, 0.f, 0.f, 0.f}, ay = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int s = 0; s < D / 32; ++s) {
            u32x4 kx = *reinterpret_cast<const u32x4*>(Ks + rx * KSTR + 32 * s + 8 * g);
            u32x4 ky = *reinterpret_cast<const u32x4*>(Ks + (rx + 4) * KSTR + 32 * s + 8 * g);
            ax = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, kx), __builtin_bit_cast(bf16x8, qreg[s]), ax, 0, 0, 0);
            ay = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, ky), __builtin_bit_cast(bf16x8, qreg[s]), ay, 0, 0, 0);
          }
          // lane holds scores of rows sb + 8g + e (e < 8) for query col
          float sv[8];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            sv[i] = (sb + 8 * g + i < re) ? ax[i] * a.scale : -INFINITY;
            sv[4 + i] = (sb + 8 * g + 4 + i < re) ? ay[i] * a.scale : -INFINITY;
          }
          float mb = sv[0];
#pragma unroll
          for (int e = 1; e < 8; ++e) mb = fmaxf(mb, sv[e]);
          mb = fmaxf(mb, __shfl_xor(mb, 16));
          mb = fmaxf(mb, __shfl_xor(mb, 32));
          const float m_new = fmaxf(m_run, mb);
          const float alpha = __expf(m_run - m_new);
          float pv[8], ps = 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            pv[e] = sv[e] > -INFINITY ? __expf(sv[e] - m_new) : 0.f;
            ps += pv[e];
          }
          ps += __shfl_xor(ps, 16);
          ps += __shfl_xor(ps, 32);
          l_run = l_run * alpha + ps;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float ai = __shfl(alpha, 4 * g + i);
#pragma unroll
            for (int cb = 0; cb < D / 16; ++cb) O[cb][i] *= ai;
          }
          u32x4 pp = {pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]),
                      pack_bf16x2(pv[4], pv[5]), pack_bf16x2(pv[6], pv[7])};
          const uint32_t* vrow = Vl + ((sb >> 1) + 4 * g) * VPS + col;
#pragma unroll
          for (int cb = 0; cb < D / 16; ++cb) {
            u32x4 vb = {vrow[cb * 16], vrow[VPS + cb * 16], vrow[2 * VPS + cb * 16],
                        vrow[3 * VPS + cb * 16]};
            O[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, pp), __builtin_bit_cast(bf16x8, vb), O[cb], 0, 0, 0);
          }
          m_run = m_new;
        }
      } else {
        const float* Kf = reinterpret_cast<const float*>(Ks);
        const float* Vf = reinterpret_cast<const float*>(Vl);
        for (int sb = rb; sb < re; sb += 16) {
          f32x4 acc = tile_dot_f32<D>(Kf + (sb + col) * KSTR,
                                      reinterpret_cast<const float*>(qrow),
                                      f32x4{0.f, 0.f, 0.f, 0.f});
          // lane holds scores of rows sb + 4g + i for query col
          float sv[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) sv[i] = (sb + 4 * g + i < re) ? acc[i] * a.scale : -INFINITY;
          float mb = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
          mb = fmaxf(mb, __shfl_xor(mb, 16));
          mb = fmaxf(mb, __shfl_xor(mb, 32));
          const float m_new = fmaxf(m_run, mb);
          const float alpha = __expf(m_run - m_new);
          float pv[4], ps = 0.f;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            pv[i] = sv[i] > -INFINITY ? __expf(sv[i] - m_new) : 0.f;
            ps += pv[i];
          }
          ps += __shfl_xor(ps, 16);
          ps += __shfl_xor(ps, 32);
          l_run = l_run * alpha + ps;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float ai = __shfl(alpha, 4 * g + i);
#pragma unroll
            for (int cb = 0; cb < D / 16; ++cb) O[cb][i] *= ai;
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) {
#pragma unroll
            for (int cb = 0; cb < D / 16; ++cb) {
              const float vb = Vf[(sb + 4 * g + i) * VPS + cb * 16 + col];
              O[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[i], vb, O[cb], 0, 0, 0);
            }
          }
          m_run = m_new;
        }
      }
    }

    if (tsplit == 1) {
      if (active) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int q = qb * 16 + 4 * g + i;
          if (q < a.B) {
#pragma unroll
            for (int cb = 0; cb < D / 16; ++cb) po_base[(long)q * D + cb * 16 + col] = O[cb][i];
          }
        }
        const int q = qb * 16 + col;
        if (g == 0 && q < a.B) {
          ps_base[q] = m_run;
          ps_base[a.B + q] = l_run;
        }
      }
    } else {
      // one group; the tsplit waves of a query block merge their row parts
      __syncthreads();
      float* cO = reinterpret_cast<float*>(smem);  // [NW][16][D]
      float* cm = cO + NW * 16 * D;                 // [NW][16]
      float* cl = cm + NW * 16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int cb = 0; cb < D / 16; ++cb)
          cO[(wave * 16 + 4 * g + i) * D + cb * 16 + col] = O[cb][i];
      }
      if (g == 0) {
        cm[wave * 16 + col] = m_run;
        cl[wave * 16 + col] = l_run;
      }
      __syncthreads();
      if (part == 0 && active) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int rr = 4 * g + i;
          const int q = qb * 16 + rr;
          float M = -INFINITY;
          for (int pp = 0; pp < tsplit; ++pp) M = fmaxf(M, cm[(wave + pp) * 16 + rr]);
          float lsum = 0.f;
          float wgt[4];
#pragma unroll
          for (int pp = 0; pp < 4; ++pp) {
            const float mp = pp < tsplit ? cm[(wave + pp) * 16 + rr] : -INFINITY;
            wgt[pp] = mp > -INFINITY ? __expf(mp - M) : 0.f;
            if (pp < tsplit) lsum += wgt[pp] * cl[(wave + pp) * 16 + rr];
          }
          if (q < a.B) {
#pragma unroll
            for (int cb = 0; cb < D / 16; ++cb) {
              float o = 0.f;
              for (int pp = 0; pp < tsplit; ++pp)
                o += wgt[pp] * cO[((wave + pp) * 16 + rr) * D + cb * 16 + col];
              po_base[(long)q * D + cb * 16 + col] = o;
            }
            if (col == 0) {
              ps_base[q] = M;
              ps_base[a.B + q] = lsum;
            }
          }
        }
      }
    }
  }
}

// ------------------------------------------------------------ bf16 ring path
//
// Chunks of kRingRows cache rows (K and V) stream into an LDS ring through
// direct global->LDS loads; rows stay in their natural row-major form with
// swizzled 16-byte granules.  The PV B operand (8 consecutive rows of one
// channel per lane) comes from two ds_read_b64_tr_b16: in each 16-lane group,
// lane i points at row t0 + i/4, channels c0 + 4(i%4) .. +3, and receives
// rows t0 .. t0+3 of channel c0 + i.
constexpr int kRingRows = 64;

typedef short v4i16 __attribute__((ext_vector_type(4)));

template <int D>
struct RingRowPtr {
  const bf16_t* base;
  const bf16_t* tail;
  const int32_t* toks;  // LDS: token ids of the split's selected rows, or null
  long unit_rows;       // rows per unit in `base`
  long r0, rlast;       // absolute first row of the chunk, last valid row
  long split_r0;        // first row of the split (toks[0])
  long Lf;              // rows Lf .. Lf + R - 1 of `base` follow the token list
  int u, nsel, G, R;
  __device__ __forceinline__ const bf16_t* operator()(int r) const {
    const long rr = min(r0 + r, rlast);
    if (toks) {
      // token ids are clamped into the unit: a bad id cannot leave K / V
      if (rr < nsel)
        return base + ((long)u * unit_rows +
                       min(max((long)toks[rr - split_r0], 0L), unit_rows - 1)) * D;
      if (rr < nsel + R) return base + ((long)u * unit_rows + Lf + (rr - nsel)) * D;
      return tail + ((long)u * G + (rr - nsel - R)) * D;
    }
    return base + ((long)u * unit_rows + rr) * D;
  }
};

// 8 waves, two per SIMD, so that one wave's MFMA, exp and LDS latencies
// overlap the other's work; with up to four query blocks each block's rows
// are split over two waves.
constexpr int kAttnRingBlock = 512;

// SEL (token-level path): the workgroup first takes the unit's top-nsel
// tokens of the scan weights itself (eq. 9 over the pool; ties to the lower
// pool position, which is the lower token) and keeps the ascending ids of
// its split; tok_out (nullable) receives them.
template <int D, bool SEL = false>
__global__ __launch_bounds__(kAttnRingBlock) void attn_ring_kernel(AttnArgs a) {
  constexpr int NW = kAttnRingBlock / kWave;
  constexpr int CR = kRingRows;
  constexpr int G = D / 8;
  constexpr int CHB = CR * 2 * D;            // bytes of one K (or V) chunk
  constexpr int IPW = CR * G / (64 * NW);    // loads per wave per matrix
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* ring = smem;                                       // [nbuf][K, V]
  int32_t* toks = reinterpret_cast<int32_t*>(smem + (size_t)a.nbuf * 2 * CHB);

  const int item = xcd_swizzle(blockIdx.x, gridDim.x);
  const int u = item / a.NS, sp = item % a.NS;
  const long rb0 = (long)sp * a.rps;
  const long re0 = min(rb0 + (long)a.rps, (long)a.nrows);
  const int nch = (int)((re0 - rb0 + CR - 1) / CR);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, col = lane & 15;

  if constexpr (SEL) {
    // the selection's histograms, the unit's region ids and (when they fit)
    // its scan weights in the ring, which is free until the first chunk
    auto& sh = *reinterpret_cast<SelectShared<kAttnRingBlock>*>(ring);
    int32_t* segl = reinterpret_cast<int32_t*>(ring + sizeof(SelectShared<kAttnRingBlock>));
    float* Wl = reinterpret_cast<float*>(segl + a.S);
    const int sel = u / a.share;  // the unit's selection
    const float* Wg = a.wpool + (long)sel * a.P;
    for (int i = threadIdx.x; i < a.S; i += kAttnRingBlock) segl[i] = a.seg[(long)sel * a.S + i];
    const long hi = min(re0, (long)a.nsel);
    const int J = a.J, mask = (1 << J) - 1;
    int32_t* tout =
        a.tok_out && u % a.share == 0 ? a.tok_out + (long)sel * a.nsel : nullptr;
    auto emit = [&](uint32_t pos, int pp) {
      if ((long)pos >= rb0 && (long)pos < hi) {
        const int32_t t = (segl[pp >> J] << J) | (pp & mask);
        toks[pos - rb0] = t;
        if (tout) tout[pos] = t;
      }
    };
    constexpr int EPT = 16;  // weights per thread held in registers
    if (a.P <= EPT * kAttnRingBlock) {
      // (the selection's first barrier publishes the region ids)
      block_select_topk_regs<kAttnRingBlock, EPT>(Wg, a.P, a.nsel, emit, sh);
    } else {
      if (a.w_in_lds) {
        for (int i = threadIdx.x; i < a.P; i += kAttnRingBlock) Wl[i] = Wg[i];
        __syncthreads();
        block_select_topk<kAttnRingBlock>(Wl, a.P, a.nsel, emit, sh);
      } else {
        __syncthreads();
        block_select_topk<kAttnRingBlock>(Wg, a.P, a.nsel, emit, sh);
      }
    }
  } else if (a.tok) {
    const long hi = min(re0, (long)a.nsel);
    for (long i = rb0 + threadIdx.x; i < hi; i += kAttnRingBlock)
      toks[i - rb0] = a.tok[(long)(u / a.share) * a.nsel + i];
  }
  __syncthreads();

  RingRowPtr<D> kp, vp;
  kp.base = reinterpret_cast<const bf16_t*>(a.K);
  vp.base = reinterpret_cast<const bf16_t*>(a.V);
  kp.tail = reinterpret_cast<const bf16_t*>(a.Kg);
  vp.tail = reinterpret_cast<const bf16_t*>(a.Vg);
  const bool indexed = SEL || a.tok != nullptr;
  kp.toks = vp.toks = indexed ? toks : nullptr;
  kp.unit_rows = vp.unit_rows = indexed ? (long)a.L : (long)a.nrows;
  kp.rlast = vp.rlast = re0 - 1;
  kp.split_r0 = vp.split_r0 = rb0;
  kp.u = vp.u = u;
  kp.nsel = vp.nsel = a.nsel;
  kp.G = vp.G = a.G;
  kp.R = vp.R = a.R;
  kp.Lf = vp.Lf = a.Lf;

  const int nqb = (a.B + 15) / 16;
  const int tsplit = 2 * nqb <= NW ? 2 : 1;  // row halves per query block
  const int qpg = NW / tsplit;
  const int ngroups = (nqb + qpg - 1) / qpg;
  const int part = wave % tsplit;
  const int R = CR / tsplit;
  const bf16_t* Qunit = reinterpret_cast<const bf16_t*>(a.Q) + (long)u * a.B * D;
  float* po_base = a.part + ((long)u * a.NS + sp) * a.B * D;
  float* ps_base = a.pstat + ((long)u * a.NS + sp) * 2 * a.B;
  const uint32_t ring_lds = lds_offset(ring);
  const int nbuf = a.nbuf;
  const float c2 = a.scale * kLog2e;  // scores in log2 units

  // K and V rows of chunk c into the ring slot at `slot`.  A chunk whose
  // rows are all selected tokens (rows past the split repeat its last row)
  // takes one token id and one address per row for both loads; any other
  // chunk goes through the general row map.
  const bf16_t* kunit = kp.base + (long)u * kp.unit_rows * D;
  const bf16_t* vunit = vp.base + (long)u * vp.unit_rows * D;
  const int split_last = (int)(re0 - 1 - rb0);
  auto issue_kv = [&](int c, uint32_t slot) {
    const long r0 = rb0 + (long)c * CR;
    if (indexed && min(r0 + CR, re0) <= (long)a.nsel) {
      constexpr int RPI = 64 / G;
      // every token id is read from LDS before the first load is issued (an
      // LDS read between two asm loads waits out its own latency each time)
      long off[IPW];
#pragma unroll
      for (int i = 0; i < IPW; ++i) {
        const int r = (wave * IPW + i) * RPI + lane / G;
        const int k = (lane % G) ^ granule_swz<G>(r);
        // token ids are clamped into the unit: a bad id cannot leave K / V
        const int t = min(max(toks[min((int)(r0 - rb0) + r, split_last)], 0), a.L - 1);
        off[i] = (long)t * D + 8 * k;
      }
#pragma unroll
      for (int i = 0; i < IPW; ++i) {
        const int inst = wave * IPW + i;
        async_load16<true>(kunit + off[i], __builtin_amdgcn_readfirstlane(slot + 1024u * inst));
        async_load16<true>(vunit + off[i], __builtin_amdgcn_readfirstlane(slot + CHB + 1024u * inst));
      }
    } else {
      kp.r0 = vp.r0 = r0;
      issue_chunk<CR, G, NW, true>(slot, kp);
      issue_chunk<CR, G, NW, true>(slot + CHB, vp);
    }
  };

  // LDS byte offsets of the lane's operands inside a 32-row block: the
  // granule swizzle depends only on the row mod 32 and every block starts at
  // a multiple of 32 rows, so one set serves all blocks
  int koff[D / 32], kyoff[D / 32], vlo[D / 16], vhi[D / 16];
  {
    const int rx0 = 8 * (col >> 2) + (col & 3);  // QK rows rx0 and rx0 + 4
    const int t00 = 8 * g + (col >> 2);          // PV rows t00 and t00 + 4
#pragma unroll
    for (int s = 0; s < D / 32; ++s) {
      koff[s] = granule_offset<G>(rx0, 4 * s + g);
      kyoff[s] = granule_offset<G>(rx0 + 4, 4 * s + g);
    }
#pragma unroll
    for (int cb = 0; cb < D / 16; ++cb) {
      const int gran = 2 * cb + ((col & 3) >> 1);
      const int byte = 8 * (col & 1);
      vlo[cb] = granule_offset<G>(t00, gran) + byte;
      vhi[cb] = granule_offset<G>(t00 + 4, gran) + byte;
    }
  }

  for (int grp = 0; grp < ngroups; ++grp) {
    const int qb = grp * qpg + wave / tsplit;
    const bool active = qb < nqb;
    const bf16_t* qrow = Qunit + (long)min(qb * 16 + col, a.B - 1) * D;
    u32x4 qreg[D / 32];
#pragma unroll
    for (int s = 0; s < D / 32; ++s)
      qreg[s] = *reinterpret_cast<const u32x4*>(qrow + 32 * s + 8 * g);
    f32x4 O[D / 16];
#pragma unroll
    for (int cb = 0; cb < D / 16; ++cb) O[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;
    // consume the q operand before async loads are queued, so that the
    // compiler's own wait for it sits here and not inside the loop below
#pragma unroll
    for (int s = 0; s < D / 32; ++s) asm volatile("" ::"v"(qreg[s]));
    // ring of nbuf slots, nbuf - 1 chunks in flight ahead of the one consumed
    for (int k = 0; k < nch && k < nbuf - 1; ++k)
      issue_kv(k, ring_lds + (uint32_t)(k * 2 * CHB));
    for (int ch = 0; ch < nch; ++ch) {
      const int nr = (int)min((long)CR, re0 - (rb0 + (long)ch * CR));
      wait_vmcnt_chunks<2 * IPW>(min(nch - 1 - ch, nbuf - 2));
      lds_barrier();  // chunk ch visible; everyone is past chunk ch - 1
      if (ch + nbuf - 1 < nch)
        issue_kv(ch + nbuf - 1, ring_lds + (uint32_t)(((ch + nbuf - 1) % nbuf) * 2 * CHB));
      const unsigned char* Kb = ring + (ch % nbuf) * 2 * CHB;
      const unsigned char* Vb = Kb + CHB;
      if (active) {
        const int rb = part * R;
        const int re = min(rb + R, nr);
        for (int sb = rb; sb < re; sb += 32) {
          // every LDS operand of the block is read first: the V reads'
          // latency then overlaps the QK products and the softmax
          const unsigned char* kblk = Kb + sb * (16 * G);
          const uint32_t vblk = lds_offset(Vb) + (uint32_t)(sb * (16 * G));
          u32x4 kx[D / 32], ky[D / 32], vb[D / 16];
#pragma unroll
          for (int s = 0; s < D / 32; ++s) {
            kx[s] = *reinterpret_cast<const u32x4*>(kblk + koff[s]);
            ky[s] = *reinterpret_cast<const u32x4*>(kblk + kyoff[s]);
          }
#pragma unroll
          for (int cb = 0; cb < D / 16; ++cb) {
            const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) v4i16*)(size_t)(vblk + vlo[cb]));
            const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) v4i16*)(size_t)(vblk + vhi[cb]));
            const u32x2 l2 = __builtin_bit_cast(u32x2, lo);
            const u32x2 h2 = __builtin_bit_cast(u32x2, hi);
            vb[cb] = u32x4{l2[0], l2[1], h2[0], h2[1]};
          }
          f32x4 ax = {0.f, 0.f, 0.f, 0.f}, ay = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int s = 0; s < D / 32; ++s) {
            ax = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, kx[s]), __builtin_bit_cast(bf16x8, qreg[s]), ax, 0, 0, 0);
            ay = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, ky[s]), __builtin_bit_cast(bf16x8, qreg[s]), ay, 0, 0, 0);
          }
          // lane holds the scores of rows sb + 8g + e (e < 8) for query col,
          // here in log2 units; rows past the range (only in a last partial
          // block) are -inf
          float t[8];
          const bool full = sb + 32 <= re;  // uniform
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            t[i] = ax[i] * c2;
            t[4 + i] = ay[i] * c2;
          }
          if (!full) {
#pragma unroll
            for (int e = 0; e < 8; ++e)
              if (sb + 8 * g + e >= re) t[e] = -INFINITY;
          }
          float mb = fmaxf(fmaxf(fmaxf(t[0], t[1]), fmaxf(t[2], t[3])),
                           fmaxf(fmaxf(t[4], t[5]), fmaxf(t[6], t[7])));
          mb = max_xor32(max_xor16(mb));
          const float m_new = fmaxf(m_run, mb);  // finite: row sb is in range
          float pv[8], ps = 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            pv[e] = __builtin_amdgcn_exp2f(t[e] - m_new);  // 2^-inf = 0
            ps += pv[e];
          }
          ps = add_xor32(add_xor16(ps));
          // rescale only when some row maximum grew: otherwise the factor
          // is exactly 1 and the update is the same without it
          if (__builtin_amdgcn_ballot_w64(m_new != m_run) != 0) {
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            l_run = l_run * alpha + ps;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float ai = __shfl(alpha, 4 * g + i);
#pragma unroll
              for (int cb = 0; cb < D / 16; ++cb) O[cb][i] *= ai;
            }
          } else {
            l_run += ps;
          }
          const u32x4 pp = {pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]),
                            pack_bf16x2(pv[4], pv[5]), pack_bf16x2(pv[6], pv[7])};
#pragma unroll
          for (int cb = 0; cb < D / 16; ++cb)
            O[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, pp), __builtin_bit_cast(bf16x8, vb[cb]), O[cb], 0, 0, 0);
          m_run = m_new;
        }
      }
    }
    lds_barrier();  // the ring is idle before it is refilled or reused

    if (tsplit == 1) {
      if (active) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int q = qb * 16 + 4 * g + i;
          if (q < a.B) {
#pragma unroll
            for (int cb = 0; cb < D / 16; ++cb) po_base[(long)q * D + cb * 16 + col] = O[cb][i];
          }
        }
        const int q = qb * 16 + col;
        if (g == 0 && q < a.B) {
          ps_base[q] = m_run * kLn2;  // back to natural-log units
          ps_base[a.B + q] = l_run;
        }
      }
    } else {
      // one group; the two waves of a query block merge their row halves
      // (the ring is idle: every wave passed the barrier after the loop)
      float* cO = reinterpret_cast<float*>(smem);  // [NW][16][D]
      float* cm = cO + NW * 16 * D;                 // [NW][16]
      float* cl = cm + NW * 16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int cb = 0; cb < D / 16; ++cb)
          cO[(wave * 16 + 4 * g + i) * D + cb * 16 + col] = O[cb][i];
      }
      if (g == 0) {
        cm[wave * 16 + col] = m_run;
        cl[wave * 16 + col] = l_run;
      }
      lds_barrier();
      if (part == 0 && active) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int rr = 4 * g + i;
          const int q = qb * 16 + rr;
          const float m0 = cm[wave * 16 + rr], m1 = cm[(wave + 1) * 16 + rr];
          const float M = fmaxf(m0, m1);
          const float w0 = m0 > -INFINITY ? __builtin_amdgcn_exp2f(m0 - M) : 0.f;
          const float w1 = m1 > -INFINITY ? __builtin_amdgcn_exp2f(m1 - M) : 0.f;
          const float lsum = w0 * cl[wave * 16 + rr] + w1 * cl[(wave + 1) * 16 + rr];
          if (q < a.B) {
#pragma unroll
            for (int cb = 0; cb < D / 16; ++cb)
              po_base[(long)q * D + cb * 16 + col] =
                  w0 * cO[(wave * 16 + rr) * D + cb * 16 + col] +
                  w1 * cO[((wave + 1) * 16 + rr) * D + cb * 16 + col];
            if (col == 0) {
              ps_base[q] = M * kLn2;  // back to natural-log units
              ps_base[a.B + q] = lsum;
            }
          }
        }
      }
    }
  }
}

// Merges the splits of each query row: O = sum_s e^(M_s - M) O_s / sum_s
// e^(M_s - M) l_s.  A workgroup takes 2048 / D rows of one unit, a thread 8
// consecutive channels of one row (two 16-byte loads per split, one 16-byte
// store for bf16).
constexpr int kCombineBlock = 256;

template <typename T>
__device__ __forceinline__ void store8(T* dst, const float* v);
template <>
__device__ __forceinline__ void store8<bf16_t>(bf16_t* dst, const float* v) {
  *reinterpret_cast<u32x4*>(dst) = u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                         pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
}
template <>
__device__ __forceinline__ void store8<float>(float* dst, const float* v) {
  reinterpret_cast<float4*>(dst)[0] = float4{v[0], v[1], v[2], v[3]};
  reinterpret_cast<float4*>(dst)[1] = float4{v[4], v[5], v[6], v[7]};
}

// Output row q, channels c0 .. c0 + 7, of unit u merged from the unit's NS
// split partials.
template <typename T>
__device__ __forceinline__ void merge_splits(const AttnArgs& a, int u, int q, int c0, int D) {
  const float* ps = a.pstat + (long)u * a.NS * 2 * a.B;
  // splits in groups of SB whose loads are all in flight together; each
  // group is merged into the running (max, sum, output) in one step, so up
  // to SB splits the arithmetic is the plain max-then-sum
  constexpr int SB = 8;
  float M = -INFINITY, lsum = 0.f;
  float o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < a.NS; s0 += SB) {
    float ms[SB], zs[SB];
    float4 x[SB][2];
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const int s = s0 + k;
      if (s < a.NS) {
        ms[k] = ps[(long)s * 2 * a.B + q];
        zs[k] = ps[(long)s * 2 * a.B + a.B + q];
        const float4* src =
            reinterpret_cast<const float4*>(a.part + (((long)u * a.NS + s) * a.B + q) * D + c0);
        x[k][0] = src[0];
        x[k][1] = src[1];
      } else {
        ms[k] = -INFINITY;
        zs[k] = 0.f;
        x[k][0] = x[k][1] = float4{0.f, 0.f, 0.f, 0.f};
      }
    }
    float mn = M;
#pragma unroll
    for (int k = 0; k < SB; ++k) mn = fmaxf(mn, ms[k]);
    if (mn == -INFINITY) continue;
    const float r = M > -INFINITY ? __expf(M - mn) : 0.f;
    lsum *= r;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] *= r;
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const float w = ms[k] > -INFINITY ? __expf(ms[k] - mn) : 0.f;
      lsum += zs[k] * w;
      o[0] += w * x[k][0].x;
      o[1] += w * x[k][0].y;
      o[2] += w * x[k][0].z;
      o[3] += w * x[k][0].w;
      o[4] += w * x[k][1].x;
      o[5] += w * x[k][1].y;
      o[6] += w * x[k][1].z;
      o[7] += w * x[k][1].w;
    }
    M = mn;
  }
  const float inv = 1.f / lsum;
#pragma unroll
  for (int i = 0; i < 8; ++i) o[i] *= inv;
  store8<T>(reinterpret_cast<T*>(a.O) + ((long)u * a.B + q) * D + c0, o);
}

template <typename T>
__global__ __launch_bounds__(kCombineBlock) void attn_combine_kernel(AttnArgs a, int D) {
  const int tpr = D / 8;                  // threads per row
  const int rpb = kCombineBlock / tpr;    // rows per workgroup
  const int nqb = (a.B + rpb - 1) / rpb;
  // the unit on the XCD whose L2 took its partials from the attention
  const int item = xcd_swizzle(blockIdx.x, gridDim.x);
  const int u = item / nqb;
  const int q = (item % nqb) * rpb + threadIdx.x / tpr;
  const int c0 = (threadIdx.x % tpr) * 8;
  if (q >= a.B) return;  // no barrier follows
  merge_splits<T>(a, u, q, c0, D);
}

// Sparse cache rows: [K[tok]; Kg] and [V[tok]; Vg], 16 bytes per thread.
__global__ __launch_bounds__(kBlock) void gather_kernel(GatherArgs a) {
  const int vpr = a.D * a.elem / 16;
  const long rows = (long)a.keff + a.R + a.G;
  const long total = (long)a.U * rows * vpr;
  for (long v = (long)blockIdx.x * kBlock + threadIdx.x; v < total;
       v += (long)gridDim.x * kBlock) {
    const long ur = v / vpr;
    const int k = (int)(v % vpr);
    const int u = (int)(ur / rows);
    const long r = ur % rows;
    const unsigned char* ks;
    const unsigned char* vs;
    const long row_bytes = (long)a.D * a.elem;
    if (r < a.keff) {
      const long t = min(max((long)a.tok[(long)u * a.keff + r], 0L), (long)a.L - 1);
      ks = (const unsigned char*)a.K + ((long)u * a.L + t) * row_bytes;
      vs = (const unsigned char*)a.V + ((long)u * a.L + t) * row_bytes;
    } else if (r < a.keff + a.R) {
      ks = (const unsigned char*)a.K + ((long)u * a.L + a.Lf + (r - a.keff)) * row_bytes;
      vs = (const unsigned char*)a.V + ((long)u * a.L + a.Lf + (r - a.keff)) * row_bytes;
    } else {
      ks = (const unsigned char*)a.Kg + ((long)u * a.G + (r - a.keff - a.R)) * row_bytes;
      vs = (const unsigned char*)a.Vg + ((long)u * a.G + (r - a.keff - a.R)) * row_bytes;
    }
    const long dst = ur * row_bytes + (long)k * 16;
    *reinterpret_cast<u32x4*>((unsigned char*)a.Ks + dst) =
        *reinterpret_cast<const u32x4*>(ks + k * 16);
    *reinterpret_cast<u32x4*>((unsigned char*)a.Vs + dst) =
        *reinterpret_cast<const u32x4*>(vs + k * 16);
  }
}

// ------------------------------------------------------------ host side

AttnPlan plan_attn(const wf_params& p, long nrows) {
  AttnPlan a{};
  const long U = (long)p.batch * p.heads;
  const int D = p.head_dim;
  if (p.dtype == WF_BF16) {
    // one workgroup per CU streaming its rows through the LDS ring
    const long chunks = std::max(1L, (nrows + kRingRows - 1) / kRingRows);
    const long want = std::max(1L, (long)(device_cu_count() + U - 1) / U);
    long splits = std::min(chunks, want);
    splits = std::max(splits, (nrows + 4095) / 4096);  // at most 4096 rows each
    const long cps = (chunks + splits - 1) / splits;
    a.rps = (int)(cps * kRingRows);
    a.splits = (int)((nrows + a.rps - 1) / a.rps);
    const size_t stage = (size_t)2 * kRingRows * 2 * D;      // K + V chunk
    const size_t toks = (size_t)a.rps * sizeof(int32_t);
    const size_t budget = 160 * 1024 - 1024;
    // three slots (two chunks in flight) measured slightly faster than four
    a.nbuf = (int)std::min<size_t>(3, (budget - toks) / stage);
    if (a.nbuf < 2) a.nbuf = 0;  // rejected by the caller
    constexpr int nw = kAttnRingBlock / kWave;  // row-half merge: [nw][16][D] + 2 [nw][16]
    const size_t comb = (size_t)nw * 16 * D * 4 + (size_t)2 * nw * 16 * 4;
    a.lds_bytes = std::max((size_t)a.nbuf * stage, comb) + toks;
    return a;
  }
  const long chunks = std::max(1L, (nrows + kAttnChunk - 1) / kAttnChunk);
  // about 512 workgroups: splits of whole chunks; every split is non-empty
  const long want = std::max(1L, (512 + U - 1) / U);
  const long splits = std::min(chunks, want);
  const long cps = (chunks + splits - 1) / splits;
  a.rps = (int)(cps * kAttnChunk);
  a.splits = (int)((nrows + a.rps - 1) / a.rps);
  const size_t stage = (size_t)kAttnChunk * (D + 4) * 4 * 2;
  const size_t comb = (size_t)4 * 16 * D * 4 + (size_t)2 * 4 * 16 * 4;
  a.lds_bytes = std::max(stage, comb);
  return a;
}

template <typename T, int D>
static hipError_t attn_launch(const AttnArgs& a, size_t lds, hipStream_t s) {
  auto kern = [] {
    if constexpr (sizeof(T) == 2) return attn_ring_kernel<D>;
    else return attn_kernel<T, D>;
  }();
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess) return e;
  }
  const int block = sizeof(T) == 2 ? kAttnRingBlock : kBlock;
  hipLaunchKernelGGL(kern, dim3((unsigned)(a.U * a.NS)), dim3(block), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_attn(const wf_params& p, const void* Q, const void* K,
                       const void* V, const int32_t* tok, int nsel,
                       const void* Kg, const void* Vg, int G, long nrows,
                       float* part, float* pstat, hipStream_t s, int share) {
  if (share < 1 || (p.batch * p.heads) % share != 0) return hipErrorInvalidValue;
  const AttnPlan pl = plan_attn(p, nrows);
  AttnArgs a;
  a.share = share;
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.tok = tok;
  a.Kg = Kg;
  a.Vg = Vg;
  a.part = part;
  a.pstat = pstat;
  a.O = nullptr;
  a.U = p.batch * p.heads;
  a.L = p.ctx_len;
  a.B = p.q_len;
  a.nsel = nsel;
  a.G = G;
  // indexed rows: the selection, then the always-kept remainder, then the tail
  a.Lf = filtered_len(p);
  a.R = tok ? (int)remainder_len(p) : 0;
  a.nrows = (int)nrows;
  a.NS = pl.splits;
  a.rps = pl.rps;
  a.nbuf = pl.nbuf;
  a.scale = effective_scale(p);
  const bool d128 = p.head_dim == 128;
  if (p.dtype == WF_BF16)
    return d128 ? attn_launch<bf16_t, 128>(a, pl.lds_bytes, s)
                : attn_launch<bf16_t, 64>(a, pl.lds_bytes, s);
  return d128 ? attn_launch<float, 128>(a, pl.lds_bytes, s)
              : attn_launch<float, 64>(a, pl.lds_bytes, s);
}

bool attn_can_select(const wf_params& p, long nrows) {
  if (p.dtype != WF_BF16 || p.segments > kSelectLdsSegs) return false;
  const AttnPlan pl = plan_attn(p, nrows);
  if (pl.nbuf < 2) return false;
  const size_t ring = (size_t)pl.nbuf * 2 * kRingRows * 2 * p.head_dim;
  return sizeof(SelectShared<kAttnRingBlock>) + (size_t)p.segments * sizeof(int32_t) <= ring;
}

hipError_t launch_attn_select(const wf_params& p, const void* Q, const void* K, const void* V,
                              const float* wpool, const int32_t* seg, int32_t* tok_out,
                              const void* Kg, const void* Vg, long nrows, float* part,
                              float* pstat, hipStream_t s, int share) {
  if (!attn_can_select(p, nrows) || share < 1 || (p.batch * p.heads) % share != 0)
    return hipErrorInvalidValue;
  const AttnPlan pl = plan_attn(p, nrows);
  AttnArgs a{};
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.tok = nullptr;
  a.wpool = wpool;
  a.seg = seg;
  a.tok_out = tok_out;
  a.Kg = Kg;
  a.Vg = Vg;
  a.part = part;
  a.pstat = pstat;
  a.share = share;
  a.U = p.batch * p.heads;
  a.L = p.ctx_len;
  a.B = p.q_len;
  a.nsel = wf_effective_budget(&p);
  a.P = p.segments << p.levels;
  a.S = p.segments;
  a.J = p.levels;
  a.G = p.gen_len;
  a.Lf = filtered_len(p);
  a.R = (int)remainder_len(p);
  a.nrows = (int)nrows;
  a.NS = pl.splits;
  a.rps = pl.rps;
  a.nbuf = pl.nbuf;
  a.scale = effective_scale(p);
  // the unit's scan weights in the ring beside the histograms and region
  // ids when they fit
  const size_t ring = (size_t)pl.nbuf * 2 * kRingRows * 2 * p.head_dim;
  const size_t fixed = sizeof(SelectShared<kAttnRingBlock>) + (size_t)a.S * sizeof(int32_t);
  a.w_in_lds = fixed + (size_t)a.P * sizeof(float) <= ring ? 1 : 0;
  auto kern = p.head_dim == 128 ? attn_ring_kernel<128, true> : attn_ring_kernel<64, true>;
  if (pl.lds_bytes > 65536) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)pl.lds_bytes);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)(a.U * a.NS)), dim3(kAttnRingBlock), pl.lds_bytes, s, a);
  return hipGetLastError();
}

hipError_t launch_attn_combine(const wf_params& p, long nrows,
                               const float* part, const float* pstat, void* O,
                               hipStream_t s) {
  AttnArgs a{};
  a.part = const_cast<float*>(part);
  a.pstat = const_cast<float*>(pstat);
  a.O = O;
  a.U = p.batch * p.heads;
  a.B = p.q_len;
  a.NS = plan_attn(p, nrows).splits;
  const int rpb = kCombineBlock / (p.head_dim / 8);
  const dim3 grid((unsigned)(a.U * ((a.B + rpb - 1) / rpb)));
  if (p.dtype == WF_BF16)
    hipLaunchKernelGGL(attn_combine_kernel<bf16_t>, grid, dim3(kCombineBlock), 0, s, a,
                       p.head_dim);
  else
    hipLaunchKernelGGL(attn_combine_kernel<float>, grid, dim3(kCombineBlock), 0, s, a,
                       p.head_dim);
  return hipGetLastError();
}

hipError_t launch_gather(const wf_params& p, const void* K, const void* V,
                         const int32_t* tok, const void* Kg, const void* Vg,
                         void* Ks, void* Vs, hipStream_t s) {
  GatherArgs a;
  a.K = K;
  a.V = V;
  a.tok = tok;
  a.Kg = Kg;
  a.Vg = Vg;
  a.Ks = Ks;
  a.Vs = Vs;
  a.U = p.batch * p.heads;
  a.L = p.ctx_len;
  a.D = p.head_dim;
  a.keff = wf_effective_budget(&p);
  a.G = p.gen_len;
  a.Lf = filtered_len(p);
  a.R = (int)remainder_len(p);
  a.elem = p.dtype == WF_BF16 ? 2 : 4;
  const long total = (long)a.U * (a.keff + a.R + a.G) * (a.D * a.elem / 16);
  const long blocks = std::min((total + kBlock - 1) / kBlock,
                               (long)device_cu_count() * 16);
  hipLaunchKernelGGL(gather_kernel, dim3((unsigned)std::max(1L, blocks)),
                     dim3(kBlock), 0, s, a);
  return hipGetLastError();
}

hipError_t load_attn_kernels() {
  hipFuncAttributes fa;
  return hipFuncGetAttributes(&fa, reinterpret_cast<const void*>(attn_ring_kernel<128, true>));
}

}  // namespace wf
