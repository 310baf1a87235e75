// Tiling-parameterised GEMM kernel family for gfx950 (CDNA4).
//
// C (M×N, fp32, row-major) = A (M×K, row-major) · B (K×N, row-major), the
// operator whose loop-tiling configuration the search tunes (§3.2, §3.3).
// A configuration's levels map to the launch as follows (level 0 outermost):
//   rows    = ((gridM·wavesM + wm)·repM + rep)·blkM + b
//   k index = ((kLoop·kSplit + z)·kSub + s)·kBlk + b
// Compile-time parameters: input dtype, MFMA size I (16/32), MFMA tiles per
// wavefront TM × TN, and the path:
//   generic — any legitimate configuration; blocks smaller than the MFMA
//             instruction are zero-padded in registers, LDS holds the natural
//             row-major tiles;
//   fast    — blocks that are multiples of the instruction: 16-byte global
//             loads staged through registers one stage ahead, B transposed in
//             registers so every LDS fragment read is one 16-byte read, LDS
//             tiles XOR-swizzled by 128-byte line to avoid bank conflicts.
// Everything else (grid, waves, block extents, stage depth, split-K, double
// buffering) is a runtime argument.
#pragma once
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <type_traits>

namespace gt {

struct KArgs {
  const void* A;
  const void* B;
  float* C;
  int64_t M, N, K;
  int32_t gridM, gridN;
  int32_t wavesM, wavesN;
  int32_t blkM, blkN;
  int32_t lgTpbM, lgTpbN;  // log2 of MFMA tiles per block (blk ≥ I) else 0
  int32_t kLoop, kSplit, kSub, kBlk;
  int32_t BM, BN, BK;
  int32_t WM, WN;          // wavefront tile
  int32_t lgBK, lgBN;
  int32_t dbuf;
  int32_t atomic;          // split-K: accumulate with fp32 atomics
  int32_t remap;           // XCD-aware workgroup order
  int32_t aVec, bVec;      // generic path: 1 or 16-byte vector tile loads
  int32_t dl;              // fast path: direct global->LDS loads into a ring
  int32_t ns;              // ring stages (direct-load path)
  int32_t aKM;             // A given K-major (K×M row-major, element (m, k) at A[k·M + m])
  int32_t lgBM;
};

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
// A 16-byte chunk as a native vector (HIP's u32x4 struct is copied by memcpy,
// which keeps staging arrays out of registers).
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <int DT>
struct Elem;
template <>
struct Elem<0> {  // fp32
  using T = float;
  static constexpr int VEC = 4;  // elements per 16-byte chunk
  static constexpr int EPL = 1;  // elements per lane per MFMA operand
};
template <>
struct Elem<1> {  // bf16 (stored as raw 16-bit patterns)
  using T = uint16_t;
  static constexpr int VEC = 8;
  static constexpr int EPL = 8;
};

template <int I>
struct AccT;
template <>
struct AccT<32> {
  using type = f32x16;
  static constexpr int N = 16;
};
template <>
struct AccT<16> {
  using type = f32x4;
  static constexpr int N = 4;
};

// Row (inside the I×I output tile) of accumulator element i held by lane;
// the column is lane % I.
template <int I>
__device__ __forceinline__ int out_row(int lane, int i) {
  if constexpr (I == 32)
    return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
  else
    return 4 * (lane >> 4) + i;
}

__device__ __forceinline__ f32x16 mfma_bf16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma_f32(float a, float b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_f32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Workgroup → (tile row, tile column). Consecutive workgroups are dispatched
// round-robin over the 8 XCDs; with `remap` each XCD receives a contiguous
// run of tiles, ordered in groups of 4 tile rows so that the tiles sharing
// an XCD's L2 share A row-blocks and B column-blocks.
__device__ __forceinline__ void tile_of(const KArgs& a, int& gm, int& gn) {
  const int nt = a.gridM * a.gridN;
  int t = static_cast<int>(blockIdx.x);
  if (a.remap) t = (t & 7) * (nt >> 3) + (t >> 3);
  constexpr int G = 4;
  const int per_group = G * a.gridN;
  const int group = t / per_group;
  const int first = group * G;
  const int gsize = min(a.gridM - first, G);
  const int r = t - group * per_group;
  gm = first + r % gsize;
  gn = r / gsize;
}

__device__ __forceinline__ void put(bool atomic, float* p, float v) {
  if (atomic)
    unsafeAtomicAdd(p, v);
  else
    *p = v;
}

// ---------------------------------------------------------------------------
// Generic path
// ---------------------------------------------------------------------------

template <typename T, int VEC>
__device__ __forceinline__ void copy_tile(T* lds, const T* g, int64_t ld, int rows, int cols,
                                          int lgcols, int vec, int tid, int nthr) {
  if (vec > 1) {
    constexpr int LGV = VEC == 8 ? 3 : 2;
    const int lgcpr = lgcols - LGV;
    const int chunks = (rows * cols) >> LGV;
    for (int e = tid; e < chunks; e += nthr) {
      const int r = e >> lgcpr;
      const int c = (e & ((1 << lgcpr) - 1)) << LGV;
      *reinterpret_cast<u32x4*>(lds + (r << lgcols) + c) =
          *reinterpret_cast<const u32x4*>(g + r * ld + c);
    }
  } else {
    const int total = rows * cols;
    for (int e = tid; e < total; e += nthr) {
      const int r = e >> lgcols;
      const int c = e & (cols - 1);
      lds[e] = g[r * ld + c];
    }
  }
}

template <int DT, int I, int TM, int TN>
__device__ void gemm_generic(const KArgs& a, char* smem) {
  using T = typename Elem<DT>::T;
  using acc_t = typename AccT<I>::type;
  constexpr int NACC = AccT<I>::N;
  constexpr int EPL = Elem<DT>::EPL;
  constexpr int G = 64 / I;
  constexpr int IK = EPL * G;
  const int tid = threadIdx.x;
  const int nthr = blockDim.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % a.wavesM;
  const int wn = wave / a.wavesM;
  int gm, gn;
  tile_of(a, gm, gn);
  const int z = blockIdx.y;

  T* As0 = reinterpret_cast<T*>(smem);
  const int stage = (a.BM + a.BN) * a.BK;
  // A K-major: the tile is BK rows of BM contiguous m, kept as [k][m] in LDS
  const bool akm = a.aKM != 0;
  const T* Ag = reinterpret_cast<const T*>(a.A) +
                (akm ? static_cast<int64_t>(gm) * a.BM : static_cast<int64_t>(gm) * a.BM * a.K);
  const T* Bg = reinterpret_cast<const T*>(a.B) + static_cast<int64_t>(gn) * a.BN;
  // LDS element offsets of A (row r, k) = r·sr + k·sk
  const int sr = akm ? 1 : a.BK, sk = akm ? a.BM : 1;

  // Rows of A / columns of B this lane feeds into each MFMA tile.
  int arow[TM], bcol[TN];
  bool aok[TM], bok[TN];
  const int tpbM = 1 << a.lgTpbM, tpbN = 1 << a.lgTpbN;
#pragma unroll
  for (int t = 0; t < TM; ++t) {
    const int in = (t & (tpbM - 1)) * I + (lane % I);
    aok[t] = in < a.blkM;
    arow[t] = wm * a.WM + (t >> a.lgTpbM) * a.blkM + in;
  }
#pragma unroll
  for (int t = 0; t < TN; ++t) {
    const int in = (t & (tpbN - 1)) * I + (lane % I);
    bok[t] = in < a.blkN;
    bcol[t] = wn * a.WN + (t >> a.lgTpbN) * a.blkN + in;
  }

  acc_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = acc_t{};

  auto load_stage = [&](int l, int buf) __attribute__((always_inline)) {
    const int64_t kbase = (static_cast<int64_t>(l) * a.kSplit + z) * a.BK;
    T* as = As0 + buf * stage;
    T* bs = as + a.BM * a.BK;
    if (akm)
      copy_tile<T, Elem<DT>::VEC>(as, Ag + kbase * a.M, a.M, a.BK, a.BM, a.lgBM, a.aVec, tid, nthr);
    else
      copy_tile<T, Elem<DT>::VEC>(as, Ag + kbase, a.K, a.BM, a.BK, a.lgBK, a.aVec, tid, nthr);
    copy_tile<T, Elem<DT>::VEC>(bs, Bg + kbase * a.N, a.N, a.BK, a.BN, a.lgBN, a.bVec, tid, nthr);
  };

  auto compute = [&](int buf) __attribute__((always_inline)) {
    const T* as = As0 + buf * stage;
    const T* bs = as + a.BM * a.BK;
    const int nkk = (a.kBlk + IK - 1) / IK;
    for (int s = 0; s < a.kSub; ++s) {
      for (int kk = 0; kk < nkk; ++kk) {
        const int kl0 = kk * IK + (lane / I) * EPL;  // this lane's first k in the sub-step
        if constexpr (DT == 1) {
          bf16x8 af[TM], bfv[TN];
#pragma unroll
          for (int t = 0; t < TM; ++t) {
            uint16_t v[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const int kl = kl0 + e;
              v[e] = (aok[t] && kl < a.kBlk) ? as[arow[t] * sr + (s * a.kBlk + kl) * sk] : uint16_t(0);
            }
            af[t] = __builtin_bit_cast(bf16x8, v);
          }
#pragma unroll
          for (int t = 0; t < TN; ++t) {
            uint16_t v[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const int kl = kl0 + e;
              v[e] = (bok[t] && kl < a.kBlk) ? bs[(s * a.kBlk + kl) * a.BN + bcol[t]] : uint16_t(0);
            }
            bfv[t] = __builtin_bit_cast(bf16x8, v);
          }
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = mfma_bf16(af[i], bfv[j], acc[i][j]);
        } else {
          float af[TM], bfv[TN];
          const bool kin = kl0 < a.kBlk;
#pragma unroll
          for (int t = 0; t < TM; ++t)
            af[t] = (aok[t] && kin) ? as[arow[t] * sr + (s * a.kBlk + kl0) * sk] : 0.0f;
#pragma unroll
          for (int t = 0; t < TN; ++t)
            bfv[t] = (bok[t] && kin) ? bs[(s * a.kBlk + kl0) * a.BN + bcol[t]] : 0.0f;
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = mfma_f32(af[i], bfv[j], acc[i][j]);
        }
      }
    }
  };

  load_stage(0, 0);
  __syncthreads();
  for (int l = 0; l < a.kLoop; ++l) {
    const int cur = a.dbuf ? (l & 1) : 0;
    const bool next = l + 1 < a.kLoop;
    if (a.dbuf && next) load_stage(l + 1, cur ^ 1);
    compute(cur);
    __syncthreads();
    if (!a.dbuf && next) {
      load_stage(l + 1, 0);
      __syncthreads();
    }
  }

  float* Cw = a.C + static_cast<int64_t>(gm) * a.BM * a.N + static_cast<int64_t>(gn) * a.BN;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
      for (int e = 0; e < NACC; ++e) {
        const int ri = (i & (tpbM - 1)) * I + out_row<I>(lane, e);
        const int ci = (j & (tpbN - 1)) * I + (lane % I);
        if (ri < a.blkM && ci < a.blkN) {
          const int r = wm * a.WM + (i >> a.lgTpbM) * a.blkM + ri;
          const int c = wn * a.WN + (j >> a.lgTpbN) * a.blkN + ci;
          put(a.atomic != 0, Cw + static_cast<int64_t>(r) * a.N + c, acc[i][j][e]);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Fast path
// ---------------------------------------------------------------------------

// 16-byte chunk q of a tile → its LDS slot: XOR inside each 128-byte line
// (8 chunks) with a hash of the line index, so that the 8 or 16 lanes served
// together by a 16-byte LDS read hit distinct banks.
__device__ __forceinline__ int swz(int q) { return q ^ (((q >> 3) ^ (q >> 6)) & 7); }

constexpr int kPfA = 8;  // A chunks staged in registers per thread
constexpr int kPfB = 1;  // B VEC×VEC blocks staged per thread

// Transpose a VEC×VEC block held as VEC row chunks into VEC column chunks.
template <int DT>
__device__ __forceinline__ void transpose_block(const u32x4* in, u32x4* out) {
  if constexpr (DT == 1) {
    // 8×8 of 16-bit values; dword w of a chunk holds elements 2w (low), 2w+1 (high)
    const uint32_t* r = reinterpret_cast<const uint32_t*>(in);  // r[j*4 + w]
    uint32_t* o = reinterpret_cast<uint32_t*>(out);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t lo = r[(2 * w) * 4 + u], hi = r[(2 * w + 1) * 4 + u];
        o[(2 * u) * 4 + w] = (lo & 0xffffu) | (hi << 16);
        o[(2 * u + 1) * 4 + w] = (lo >> 16) | (hi & 0xffff0000u);
      }
    }
  } else {
    const float* r = reinterpret_cast<const float*>(in);
    float* o = reinterpret_cast<float*>(out);
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int j = 0; j < 4; ++j) o[t * 4 + j] = r[j * 4 + t];
  }
}

template <int V>
constexpr int ilog2c() {
  return V <= 1 ? 0 : 1 + ilog2c<V / 2>();
}

// CPR = 16-byte chunks per LDS row = BK / VEC, a compile-time constant so
// that the chunk-step loop unrolls: the fragments of chunk-step cs+1 are read
// from LDS while the MFMAs of chunk-step cs run.
// AK: A given K-major; its tile is loaded like B's (VEC×VEC blocks,
// transposed in registers) into the same [m][k-chunk] LDS layout.
template <int DT, int I, int TM, int TN, int CPR, bool AK = false>
__device__ void gemm_fast(const KArgs& a, char* smem) {
  using T = typename Elem<DT>::T;
  using acc_t = typename AccT<I>::type;
  constexpr int NACC = AccT<I>::N;
  constexpr int VEC = Elem<DT>::VEC;
  constexpr int LGV = VEC == 8 ? 3 : 2;
  constexpr int G = 64 / I;          // lane groups of an MFMA operand
  constexpr int NCS = CPR / G;       // chunk-steps per stage
  constexpr int LGCPR = ilog2c<CPR>();
  constexpr int NLINE = CPR >= 8 ? CPR / 8 : 1;  // 128-byte lines per LDS row
  static_assert(NCS >= 1, "stage shallower than one MFMA K step");
  const int tid = threadIdx.x;
  const int nthr = blockDim.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % a.wavesM;
  const int wn = wave / a.wavesM;
  int gm, gn;
  tile_of(a, gm, gn);
  const int z = blockIdx.y;

  const int achunks = a.BM << LGCPR;
  const int lgnbn = a.lgBN - LGV;    // B blocks along n = BN / VEC
  const int bblocks = CPR << lgnbn;  // CPR blocks along k
  const int stage = achunks + (a.BN << LGCPR);  // chunks per stage
  u32x4* lds = reinterpret_cast<u32x4*>(smem);

  const T* Ag = reinterpret_cast<const T*>(a.A) +
                (AK ? static_cast<int64_t>(gm) * a.BM : static_cast<int64_t>(gm) * a.BM * a.K);
  const T* Bg = reinterpret_cast<const T*>(a.B) + static_cast<int64_t>(gn) * a.BN;

  const int rounds = max((achunks + nthr * kPfA - 1) / (nthr * kPfA),
                         (bblocks + nthr * kPfB - 1) / (nthr * kPfB));
  const bool prefetch = rounds == 1;

  // This thread's chunks: A chunk i is e_i = ta + i·nthr with ta = tid, i.e.
  // row (ta >> LGCPR) + i·(nthr >> LGCPR), column chunk ta & (CPR − 1), so
  // one base offset and a uniform row stride address all of them. Tile and
  // thread counts are powers of two: either every thread owns na chunks, or
  // the tile has fewer chunks than threads, na = 1 and the surplus threads
  // take the last chunk (ta clamped) and later write those same bytes to
  // its slot. The loads therefore sit under wavefront-uniform conditions only.
  const int na = __builtin_amdgcn_readfirstlane(min(kPfA, (achunks + nthr - 1) / nthr));
  const int nbb = __builtin_amdgcn_readfirstlane(min(kPfB, (bblocks + nthr - 1) / nthr));
  const int ta = min(tid, achunks - 1);
  const int64_t aoff0 = static_cast<int64_t>(ta >> LGCPR) * a.K + ((ta & (CPR - 1)) << LGV);
  const int64_t astride = static_cast<int64_t>(nthr >> LGCPR) * a.K;
  int64_t boff[kPfB];
  int bq0[kPfB];
#pragma unroll
  for (int i = 0; i < kPfB; ++i) {
    const int b = min(tid + i * nthr, bblocks - 1);
    const int nb = b & ((1 << lgnbn) - 1), kb = b >> lgnbn;
    boff[i] = static_cast<int64_t>(kb << LGV) * a.N + (nb << LGV);
    bq0[i] = ((nb << LGV) << LGCPR) + kb;
  }

  // K-major A: blocks of VEC k-rows × VEC m (one 16-byte chunk per row),
  // kPfA / VEC of them per thread in the staging registers
  constexpr int kPfAB = kPfA / VEC;
  const int lgnbm = a.lgBM - LGV;
  const int ablocks = CPR << lgnbm;
  const int nab = __builtin_amdgcn_readfirstlane(min(kPfAB, (ablocks + nthr - 1) / nthr));
  int64_t aoffk[kPfAB > 0 ? kPfAB : 1];
  int aq0[kPfAB > 0 ? kPfAB : 1];
  if constexpr (AK) {
#pragma unroll
    for (int i = 0; i < kPfAB; ++i) {
      const int b = min(tid + i * nthr, ablocks - 1);
      const int nm = b & ((1 << lgnbm) - 1), kb = b >> lgnbm;
      aoffk[i] = static_cast<int64_t>(kb << LGV) * a.M + (nm << LGV);
      aq0[i] = ((nm << LGV) << LGCPR) + kb;
    }
  }

  u32x4 ra[kPfA];
  u32x4 rb[kPfB * VEC];

  auto gload = [&](int l) __attribute__((always_inline)) {
    const int64_t kbase = (static_cast<int64_t>(l) * a.kSplit + z) * a.BK;
    const T* bg = Bg + kbase * a.N;
    if constexpr (AK) {
      const T* ag = Ag + kbase * a.M;
#pragma unroll
      for (int i = 0; i < kPfAB; ++i)
        if (i < nab) {
#pragma unroll
          for (int j = 0; j < VEC; ++j)
            ra[i * VEC + j] = *reinterpret_cast<const u32x4*>(ag + aoffk[i] + j * a.M);
        }
    } else {
      const T* ag = Ag + kbase + aoff0;
#pragma unroll
      for (int i = 0; i < kPfA; ++i)
        if (i < na) ra[i] = *reinterpret_cast<const u32x4*>(ag + i * astride);
    }
#pragma unroll
    for (int i = 0; i < kPfB; ++i)
      if (i < nbb) {
#pragma unroll
        for (int j = 0; j < VEC; ++j)
          rb[i * VEC + j] = *reinterpret_cast<const u32x4*>(bg + boff[i] + j * a.N);
      }
  };

  auto lstore = [&](int buf) __attribute__((always_inline)) {
    u32x4* as = lds + buf * stage;
    u32x4* bs = as + achunks;
    if constexpr (AK) {
#pragma unroll
      for (int i = 0; i < kPfAB; ++i)
        if (i < nab) {
          u32x4 t[VEC];
          transpose_block<DT>(&ra[i * VEC], t);
#pragma unroll
          for (int j = 0; j < VEC; ++j) as[swz(aq0[i] + (j << LGCPR))] = t[j];
        }
    } else {
#pragma unroll
      for (int i = 0; i < kPfA; ++i)
        if (i < na) as[swz(ta + i * nthr)] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < kPfB; ++i)
      if (i < nbb) {
        u32x4 t[VEC];
        transpose_block<DT>(&rb[i * VEC], t);
#pragma unroll
        for (int j = 0; j < VEC; ++j) bs[swz(bq0[i] + (j << LGCPR))] = t[j];
      }
  };

  // Tiles larger than the staging registers: load and store in rounds.
  auto load_rounds = [&](int l, int buf) __attribute__((always_inline)) {
    const int64_t kbase = (static_cast<int64_t>(l) * a.kSplit + z) * a.BK;
    u32x4* as = lds + buf * stage;
    u32x4* bs = as + achunks;
    if constexpr (AK) {
      for (int b = tid; b < ablocks; b += nthr) {
        const int nm = b & ((1 << lgnbm) - 1), kb = b >> lgnbm;
        const T* src = Ag + (kbase + (kb << LGV)) * a.M + (nm << LGV);
        u32x4 r[VEC], t[VEC];
#pragma unroll
        for (int j = 0; j < VEC; ++j) r[j] = *reinterpret_cast<const u32x4*>(src + j * a.M);
        transpose_block<DT>(r, t);
#pragma unroll
        for (int j = 0; j < VEC; ++j) as[swz((((nm << LGV) + j) << LGCPR) + kb)] = t[j];
      }
    } else {
      for (int e = tid; e < achunks; e += nthr)
        as[swz(e)] = *reinterpret_cast<const u32x4*>(
            Ag + static_cast<int64_t>(e >> LGCPR) * a.K + kbase + ((e & (CPR - 1)) << LGV));
    }
    for (int b = tid; b < bblocks; b += nthr) {
      const int nb = b & ((1 << lgnbn) - 1), kb = b >> lgnbn;
      const T* src = Bg + (kbase + (kb << LGV)) * a.N + (nb << LGV);
      u32x4 r[VEC], t[VEC];
#pragma unroll
      for (int j = 0; j < VEC; ++j) r[j] = *reinterpret_cast<const u32x4*>(src + j * a.N);
      transpose_block<DT>(r, t);
#pragma unroll
      for (int j = 0; j < VEC; ++j) bs[swz((((nb << LGV) + j) << LGCPR) + kb)] = t[j];
    }
  };

  acc_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = acc_t{};

  // Fragment addressing. Row r, chunk ch = cs·G + grp sits at slot
  // swz(r·CPR + ch) = ((X_j ^ (cs·G & 7)) + (cs·G & ~7)) with
  // X_j = swz(r·CPR + grp + 8j) − 8j for line j = (cs·G) / 8 of the row.
  const int grp = lane / I;
  int xa[TM][NLINE], xb[TN][NLINE];
#pragma unroll
  for (int t = 0; t < TM; ++t)
#pragma unroll
    for (int j = 0; j < NLINE; ++j) {
      const int q0 = ((wm * a.WM + t * I + (lane % I)) << LGCPR) + grp + 8 * j;
      xa[t][j] = swz(q0) - 8 * j;
    }
#pragma unroll
  for (int t = 0; t < TN; ++t)
#pragma unroll
    for (int j = 0; j < NLINE; ++j) {
      const int q0 = ((wn * a.WN + t * I + (lane % I)) << LGCPR) + grp + 8 * j;
      xb[t][j] = swz(q0) - 8 * j;
    }

  u32x4 fa[2][TM], fb[2][TN];
  auto load_frags = [&](const u32x4* as, int cs, int slot) __attribute__((always_inline)) {
    const u32x4* bs = as + achunks;
    const int c = cs * G;
    const int j = CPR >= 8 ? (c >> 3) : 0;
#pragma unroll
    for (int t = 0; t < TM; ++t) fa[slot][t] = as[(xa[t][j] ^ (c & 7)) + (c & ~7)];
#pragma unroll
    for (int t = 0; t < TN; ++t) fb[slot][t] = bs[(xb[t][j] ^ (c & 7)) + (c & ~7)];
  };
  auto mfmas = [&](int slot) __attribute__((always_inline)) {
    if constexpr (DT == 1) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = mfma_bf16(__builtin_bit_cast(bf16x8, fa[slot][i]),
                                __builtin_bit_cast(bf16x8, fb[slot][j]), acc[i][j]);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = mfma_f32(__builtin_bit_cast(f32x4, fa[slot][i])[q],
                                 __builtin_bit_cast(f32x4, fb[slot][j])[q], acc[i][j]);
    }
  };

  auto compute = [&](const u32x4* as) __attribute__((always_inline)) {
#pragma unroll
    for (int cs = 0; cs < NCS; ++cs) {
      if (cs + 1 < NCS) load_frags(as, cs + 1, (cs + 1) & 1);
      mfmas(cs & 1);
    }
  };

  // Main loop: every stage but the last is one straight-line block — the
  // next stage's global loads, this stage's LDS fragments and MFMAs, the
  // next stage's LDS stores — so the scheduler can interleave them.
  auto main_loop = [&](auto dbuf_tag) __attribute__((always_inline)) {
    constexpr bool DB = decltype(dbuf_tag)::value;
    gload(0);
    lstore(0);
    __syncthreads();
    load_frags(lds, 0, 0);
    int l = 0;
    for (; l + 1 < a.kLoop; ++l) {
      const int cur = DB ? (l & 1) : 0;
      const int nxt = DB ? (cur ^ 1) : 0;
      gload(l + 1);
      // keep the next stage's loads ahead of this stage's MFMAs
      __builtin_amdgcn_sched_barrier(0);
      compute(lds + cur * stage);
      if constexpr (!DB) __syncthreads();
      lstore(nxt);
      __syncthreads();
      load_frags(lds + nxt * stage, 0, 0);
    }
    compute(lds + (DB ? (l & 1) : 0) * stage);
  };

  if (prefetch) {
    if (a.dbuf)
      main_loop(std::true_type{});
    else
      main_loop(std::false_type{});
  } else {
    load_rounds(0, 0);
    __syncthreads();
    load_frags(lds, 0, 0);
    for (int l = 0; l < a.kLoop; ++l) {
      const int cur = a.dbuf ? (l & 1) : 0;
      compute(lds + cur * stage);
      if (l + 1 < a.kLoop) {
        if (!a.dbuf) __syncthreads();
        const int nxt = a.dbuf ? (cur ^ 1) : 0;
        load_rounds(l + 1, nxt);
        __syncthreads();
        load_frags(lds + nxt * stage, 0, 0);
      }
    }
  }

  float* Cw = a.C + static_cast<int64_t>(gm) * a.BM * a.N + static_cast<int64_t>(gn) * a.BN;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
      for (int e = 0; e < NACC; ++e) {
        const int r = wm * a.WM + i * I + out_row<I>(lane, e);
        const int c = wn * a.WN + j * I + (lane % I);
        put(a.atomic != 0, Cw + static_cast<int64_t>(r) * a.N + c, acc[i][j][e]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Fast path with direct global→LDS loads (bf16)
// ---------------------------------------------------------------------------
//
// Each global_load_lds_dwordx4 of a wavefront writes 64 consecutive 16-byte
// LDS slots (lane j → slot base + j) from 64 per-lane global addresses, so
// tiles reach LDS without passing through registers and a ring of ns stages
// keeps ns − 1 stages of loads in flight. A sits in LDS as [m][k] chunks,
// XOR-swizzled by swz(); with 16×16 MFMA and stages of two or more
// chunk-steps (64- and 128-deep) it is split into planes instead, one per
// chunk-step: plane cs holds the G = 4 chunks that step reads of every one of
// the BM rows, as [m][4] swizzled by swz(). Each fragment read then covers
// one aligned 1 KiB block, which the 16-byte LDS reads serve without bank
// conflicts; the stage-wide layout conflicts 2-way at those depths (with
// 32×32 MFMA, or 32-deep stages, it does not, and is kept). B stays [k][n]
// with the chunks of row k XOR-ed by bswz(k), and its MFMA operands are read
// with the transposing LDS read: inside a 16-lane group, lane l receives
// element (l & 3) of the 8 bytes addressed by lane 4j + (l >> 2) as its j-th
// value, so lanes addressing rows k0 + (i >> 2), columns n0 + 4(i & 3) hand
// lane l four consecutive k of column n0 + l.

typedef short s16x4 __attribute__((ext_vector_type(4)));
// Direct-load instructions per wavefront and stage the kernel keeps offsets
// for: 8 where the accumulator size admits 8 wavefronts (the register budget
// per lane is then 256), 16 otherwise.
constexpr int dl_inst_cap(int64_t acc) { return acc + 96 <= 256 ? 8 : 16; }

// XOR applied to the 16-byte chunk index of B row k in LDS. A transposing
// read touches rows k0 … k0+3 (k0 ≡ 0 mod 4) and, per 16-lane group, two
// adjacent chunks (four per 32 lanes with 32×32 MFMA; with 16×16 MFMA the
// second 16-lane group reads rows k0+8 … k0+11 instead). f(k mod 4) ∈
// {0, 6, 10, 12}, XOR-ed with 8 when bit 3 of k is set, sends those accesses
// to distinct 16-byte bank slots mod 128 B (16 lanes) and mod 256 B (32 lanes).
__device__ __forceinline__ int bswz(int k, int cprb) {
  const int j = k & 3;
  return (((j << 2) | (((j ^ (j >> 1)) & 1) << 1)) ^ (((k >> 3) & 1) << 3)) & (cprb - 1);
}

// vmcnt field of s_waitcnt on gfx9: bits [3:0] and [15:14]; lgkmcnt [11:8], expcnt [6:4].
template <int N>
__device__ __forceinline__ void waitcnt_vm() {
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

__device__ __forceinline__ void waitcnt_lgkm0() {
  __builtin_amdgcn_s_waitcnt(0xf | (0x3 << 14) | (0x7 << 4));  // lgkmcnt(0) only
}

// s_waitcnt takes its count as an immediate: wait for the largest of
// {0, 1, 2, 3, 4, 6, 8, 12, 16, 24, 32, 48} that is at most n (a uniform
// value), chosen by a balanced comparison tree.
__device__ __forceinline__ void wait_vm_at_most(int n) {
  if (n >= 12) {
    if (n >= 24) {
      if (n >= 48) waitcnt_vm<48>();
      else if (n >= 32) waitcnt_vm<32>();
      else waitcnt_vm<24>();
    } else {
      if (n >= 16) waitcnt_vm<16>();
      else waitcnt_vm<12>();
    }
  } else if (n >= 4) {
    if (n >= 8) waitcnt_vm<8>();
    else if (n >= 6) waitcnt_vm<6>();
    else waitcnt_vm<4>();
  } else {
    if (n >= 2) {
      if (n >= 3) waitcnt_vm<3>();
      else waitcnt_vm<2>();
    } else if (n >= 1) {
      waitcnt_vm<1>();
    } else {
      waitcnt_vm<0>();
    }
  }
}

// One 16-byte-per-lane direct global→LDS load: lane j reads 16 bytes at
// base + off (base uniform, off this lane's byte offset) and writes them to
// LDS byte address lds_base + 16·j. Written as inline assembly so that the
// compiler does not see an LDS write it would have to wait for before every
// LDS read (it cannot tell the ring slots apart); the ring's vmcnt accounting
// is done explicitly.
__device__ __forceinline__ void dma_load16(uint32_t off, uint64_t base, uint32_t lds_base) {
  // base and lds_base are uniform; reading them from the first lane keeps
  // them in scalar registers whatever the compiler inferred
  const uint64_t sb =
      static_cast<uint64_t>(static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(base)))) |
      (static_cast<uint64_t>(static_cast<uint32_t>(
           __builtin_amdgcn_readfirstlane(static_cast<int>(base >> 32))))
       << 32);
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(off), "s"(sb), "s"(__builtin_amdgcn_readfirstlane(static_cast<int>(lds_base)))
               : "memory", "m0");
}

// A wavefront-uniform pointer as a 64-bit scalar (each half taken from the
// first active lane and zero-extended).
__device__ __forceinline__ uint64_t uniform_ptr(const void* p) {
  const uint64_t b = reinterpret_cast<uintptr_t>(p);
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b)));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b >> 32)));
  return static_cast<uint64_t>(lo) | (static_cast<uint64_t>(hi) << 32);
}

// Byte offset inside LDS of a pointer into the kernel's dynamic LDS.
__device__ __forceinline__ uint32_t lds_off(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(
      (const __attribute__((address_space(3))) char*)(p)));
}

template <int I, int TM, int TN, int CPR>
__device__ __forceinline__ void gemm_fast_dl(const KArgs& a, char* smem) {
  using T = uint16_t;
  using acc_t = typename AccT<I>::type;
  constexpr int NACC = AccT<I>::N;
  constexpr int G = 64 / I;
  constexpr int NCS = CPR / G;
  constexpr int LGCPR = ilog2c<CPR>();
  constexpr int NLINE = CPR >= 8 ? CPR / 8 : 1;
  static_assert(NCS >= 1, "stage shallower than one MFMA K step");
  constexpr int kMaxDlInst = dl_inst_cap(TM * TN * I * I / 64);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nw = blockDim.x >> 6;
  const int wm = wave % a.wavesM;
  const int wn = wave / a.wavesM;
  int gm, gn;
  tile_of(a, gm, gn);
  const int z = blockIdx.y;

  const int BM = a.BM, BN = a.BN, BK = a.BK;
  const int cprb = BN >> 3;                 // 16-byte chunks per B row
  const int achunks = BM << LGCPR;
  const int bchunks = BK * cprb;
  const int stage = achunks + bchunks;      // 16-byte slots per stage
  const int pa = achunks >> 6, pb = bchunks >> 6;
  const int ninst = (pa + pb) / nw;         // load instructions per wavefront per stage
  const int ns = a.ns;
  u32x4* lds = reinterpret_cast<u32x4*>(smem);
  const T* Ag = reinterpret_cast<const T*>(a.A) + static_cast<int64_t>(gm) * BM * a.K;
  const T* Bg = reinterpret_cast<const T*>(a.B) + static_cast<int64_t>(gn) * BN;

  // Load instruction p of a stage fills slots p·64 … p·64+63; wavefront w
  // issues p = w, w + nw, … (A instructions first, then B). Each lane works
  // out the chunk its slot holds: A slot s holds chunk swz(s) (swz is an
  // involution) of the [m][k] layout, or in the plane layout chunk-step
  // s / (4·BM) and in-plane chunk swz(s mod 4·BM) of its [m][4]; B slot
  // (k, cs) holds row k, chunk cs ^ bswz(k). The lane's byte offset from the
  // stage's A (or B) origin is the same for every stage, so it is computed
  // once (it fits 32 bits: BM·K and BK·N are below 2^31).
  constexpr bool PLANES = I == 16 && NCS >= 2;
  const int lgcprb = a.lgBN - 3;
  const int na_w = pa / nw;
  uint32_t doff[kMaxDlInst];
#pragma unroll
  for (int i = 0; i < kMaxDlInst; ++i) {
    doff[i] = 0;
    if (i < na_w) {
      if constexpr (PLANES) {
        const int s = ((wave + i * nw) << 6) + lane;
        const int lgp = a.lgBM + 2;  // slots per plane: BM·4
        const int q = swz(s & ((1 << lgp) - 1));
        doff[i] = (static_cast<uint32_t>(q >> 2) * static_cast<uint32_t>(a.K) +
                   static_cast<uint32_t>((((s >> lgp) << 2) + (q & 3)) << 3)) * 2u;
      } else {
        const int q = swz(((wave + i * nw) << 6) + lane);
        doff[i] = (static_cast<uint32_t>(q >> LGCPR) * static_cast<uint32_t>(a.K) +
                   static_cast<uint32_t>((q & (CPR - 1)) << 3)) * 2u;
      }
    } else if (i < ninst) {
      const int sidx = ((wave + (i - na_w) * nw) << 6) + lane;
      const int k = sidx >> lgcprb, cs = sidx & (cprb - 1);
      doff[i] = (static_cast<uint32_t>(k) * static_cast<uint32_t>(a.N) +
                 static_cast<uint32_t>((cs ^ bswz(k, cprb)) << 3)) * 2u;
    }
  }
  const int lds0 = __builtin_amdgcn_readfirstlane(static_cast<int>(lds_off(lds)));
  const uint32_t stage16 = static_cast<uint32_t>(stage) * 16u;  // bytes per ring slot
  // bytes between the A (B) origins of consecutive stages of this split-K slice
  const uint64_t stepA = static_cast<uint64_t>(a.kSplit) * static_cast<uint64_t>(BK) * 2u;
  const uint64_t stepB = stepA * static_cast<uint64_t>(a.N);
  // Instruction i (< ninst) of this wavefront for stage l into ring slot
  // `slot`; ga, gb: the stage's A and B origins as uniform scalars.
  // A or B is picked with scalar selects, not branches.
  auto dma = [&](uint64_t ga, uint64_t gb, uint32_t sbase, int i) __attribute__((always_inline)) {
    const bool isa = i < na_w;
    const uint32_t da = static_cast<uint32_t>(wave + i * nw) * 1024u;
    const uint32_t db = static_cast<uint32_t>(achunks + ((wave + (i - na_w) * nw) << 6)) * 16u;
    dma_load16(doff[i], isa ? ga : gb, sbase + (isa ? da : db));
  };
  // Uniform origins of stage l's A and B tiles and LDS byte base of ring slot `slot`.
  struct StageBase {
    uint64_t ga, gb;
    uint32_t sb;
  };
  auto stage_base = [&](int l, int slot) __attribute__((always_inline)) {
    const int64_t kbase = (static_cast<int64_t>(l) * a.kSplit + z) * BK;
    StageBase r;
    r.ga = uniform_ptr(Ag + kbase);
    r.gb = uniform_ptr(Bg + kbase * a.N);
    r.sb = static_cast<uint32_t>(
        __builtin_amdgcn_readfirstlane(static_cast<int>(lds0 + slot * stage * 16)));
    return r;
  };
  // All of this wavefront's instructions of stage l, back to back.
  auto issue = [&](int l, int slot) __attribute__((always_inline)) {
    const StageBase b = stage_base(l, slot);
#pragma unroll
    for (int i = 0; i < kMaxDlInst; ++i)
      if (i < ninst) dma(b.ga, b.gb, b.sb, i);
  };

  acc_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = acc_t{};

  // A fragment slots: in the [m][k] layout as in the register-staged path;
  // in the plane layout, this lane's slot in plane 0 (plane cs adds 4·BM·cs).
  const int grp = lane / I;
  int xa[TM][NLINE];
#pragma unroll
  for (int t = 0; t < TM; ++t)
#pragma unroll
    for (int j = 0; j < NLINE; ++j) {
      if constexpr (PLANES) {
        xa[t][j] = swz(((wm * a.WM + t * I + (lane % I)) << 2) + grp);
      } else {
        const int q0 = ((wm * a.WM + t * I + (lane % I)) << LGCPR) + grp + 8 * j;
        xa[t][j] = swz(q0) - 8 * j;
      }
    }
  const int plane_slots = BM << 2;
  // B operand addressing: in 16-lane group g16, input lane i covers row
  // k0 + (i >> 2) (+4 for the second read), columns n0 + 4(i & 3).
  const int i16 = lane & 15, g16 = lane >> 4;
  const int kgrp = I == 32 ? (g16 >> 1) : g16;           // which 8-k group of the step
  const int ncol0 = (I == 32 ? 16 * (g16 & 1) : 0) + 4 * (i16 & 3);
  int bcol[TN];
#pragma unroll
  for (int t = 0; t < TN; ++t) bcol[t] = wn * a.WN + t * I + ncol0;  // column of this lane's 4 values
  const int krow_l = kgrp * 8 + (i16 >> 2);

  u32x4 fa[2][TM];
  u32x4 fb[2][TN];
  auto load_frags = [&](const u32x4* as, int cs, int fs) __attribute__((always_inline)) {
    const int c = cs * G;
    const int j = CPR >= 8 ? (c >> 3) : 0;
#pragma unroll
    for (int t = 0; t < TM; ++t) {
      if constexpr (PLANES)
        fa[fs][t] = as[cs * plane_slots + xa[t][0]];
      else
        fa[fs][t] = as[(xa[t][j] ^ (c & 7)) + (c & ~7)];
    }
    const char* bs = reinterpret_cast<const char*>(as + achunks);
#pragma unroll
    for (int t = 0; t < TN; ++t) {
      s16x4 h[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int k = cs * (G * 8) + krow_l + 4 * hh;
        const int col = bcol[t];
        const int chunk = (col >> 3) ^ bswz(k, cprb);
        const char* addr = bs + (k * cprb + chunk) * 16 + (col & 4) * 2;
        h[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4*)(addr));
      }
      fb[fs][t] = __builtin_bit_cast(u32x4, __builtin_shufflevector(h[0], h[1], 0, 1, 2, 3, 4, 5, 6, 7));
    }
  };
  auto mfma1 = [&](int fs, int q) __attribute__((always_inline)) {
    const int i = q / TN, j = q % TN;
    acc[i][j] = mfma_bf16(__builtin_bit_cast(bf16x8, fa[fs][i]),
                          __builtin_bit_cast(bf16x8, fb[fs][j]), acc[i][j]);
  };

  // Ring schedule. Stage s is loaded into slot s mod ns. Its loads are issued
  // in a window of NCS chunk-steps of MFMAs: the last chunk-step of stage
  // s − ns (which runs after the barrier that ends stage s − ns, once every
  // wavefront has stopped reading slot s mod ns) and chunk-steps 0 … NCS−2 of
  // stage s − ns + 1, so the whole set is out before the boundary that ends
  // stage s − ns + 1. Inside the window the wavefront's ninst instructions go
  // one at a time, one after every R-th MFMA: a wavefront waiting for room in
  // the memory pipeline cannot issue MFMAs, so loads go out in small doses,
  // and the last of them leaves half a chunk-step before the window closes.
  // Stages 0 … ns−2 (and the part of stage ns − 1's window that would precede
  // stage 0) are issued up front. The boundary (wait for stage l + 1, barrier,
  // first fragments of stage l + 1) sits in front of stage l's last
  // chunk-step of MFMAs.
  constexpr int TMTN = TM * TN;
  constexpr int SPOS = NCS * TMTN;  // MFMA slots in a window
  // The loop is instantiated for NI = cap and cap/2 instructions per
  // wavefront and stage (NI = 0: any other count, guarded per load), so the
  // common cases carry no per-load branch. Load i of a window goes after MFMA
  // slot i·R + R − 1 (slots past the window go out with its last slot). With
  // the full cap (the 64-deep stages of a two-slot ring, where a load has at
  // most one stage to land) the loads go out back to back from the window's
  // start (R = 1); with half the cap (the shallower stages of deeper rings)
  // they are spread over the first half of the window; otherwise they end
  // half a chunk-step before it closes. Measured at 4096³: front-loading
  // gains 3 % on the two-slot rings, spreading 3 % on the five-slot rings.
  // Both parts of every window use the same R.
  auto run = [&](auto ni) __attribute__((always_inline)) {
    constexpr int NI = decltype(ni)::value;
    constexpr int NIE = NI ? NI : kMaxDlInst;
    constexpr int RR = NI == kMaxDlInst ? 1 : (NI ? (SPOS / 2) / (NI ? NI : 1) : (SPOS - TMTN / 2) / NIE);
    constexpr int R = RR > 1 ? RR : 1;
    // open: the window is open for every load of this stage (no guard on it)
    auto dma_at = [&](const StageBase& sb, bool on, int pos, auto open) __attribute__((always_inline)) {
      constexpr bool OPEN = decltype(open)::value;
      const int i = pos / R;
      if (pos % R == R - 1 && i < NIE && i * R + R - 1 < SPOS) {
        if ((OPEN || on) && (NI > 0 || i < ninst)) {
          __builtin_amdgcn_sched_barrier(0);
          dma(sb.ga, sb.gb, sb.sb, i);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      if (pos == SPOS - 1) {
#pragma unroll
        for (int j = SPOS / R; j < NIE; ++j)
          if ((OPEN || on) && (NI > 0 || j < ninst)) dma(sb.ga, sb.gb, sb.sb, j);
      }
    };
    const int npro = min(ns - 1, a.kLoop);
    for (int l = 0; l < npro; ++l) issue(l, l);
    wait_vm_at_most(__builtin_amdgcn_readfirstlane((npro - 1) * ninst));
    __builtin_amdgcn_s_barrier();
    if (ns - 1 < a.kLoop) {
      // the part of stage ns − 1's window before stage 0 (slot ns − 1 is unused so far)
      const StageBase sb0 = stage_base(ns - 1, ns - 1);
#pragma unroll
      for (int pos = 0; pos < TMTN; ++pos) dma_at(sb0, true, pos, std::true_type{});
    }
    load_frags(lds, 0, 0);
    // One stage; OPEN: both windows it touches are open (all but the last ns stages).
    // cur = l mod ns and its LDS byte address cur_b, and the global origins
    // (ga2, gb2) of stage l + ns, are carried from stage to stage.
    auto stage_step = [&](int l, int cur, uint32_t cur_b, uint64_t ga2, uint64_t gb2,
                          auto open) __attribute__((always_inline)) {
      constexpr bool OPEN = decltype(open)::value;
      const u32x4* as = reinterpret_cast<const u32x4*>(smem + (cur_b - lds0));
      const int ld = l + ns - 1;  // stage whose window ends with this stage's boundary
      const bool load = OPEN || ld < a.kLoop;
      StageBase sbs{0, 0, 0};
      if (load && NCS > 1)  // stage l + ns − 1 goes into slot (cur − 1) mod ns
        sbs = StageBase{ga2 - stepA, gb2 - stepB, cur == 0 ? lds0 + (ns - 1) * stage16 : cur_b - stage16};
#pragma unroll
      for (int cs = 0; cs + 1 < NCS; ++cs) {
        load_frags(as, cs + 1, (cs + 1) & 1);
#pragma unroll
        for (int q = 0; q < TMTN; ++q) {
          mfma1(cs & 1, q);
          dma_at(sbs, load, TMTN + cs * TMTN + q, open);
        }
      }
      const bool more = OPEN || l + 1 < a.kLoop;
      const uint32_t nx_b = cur + 1 == ns ? lds0 : cur_b + stage16;
      const u32x4* nx = reinterpret_cast<const u32x4*>(smem + (nx_b - lds0));
      if (more) {
        // stages issued after stage l + 1: l + 2 … min(l + ns − 1, kLoop − 1)
        const int pending = OPEN ? ns - 2 : min(ns - 2, a.kLoop - 2 - l);
        wait_vm_at_most(__builtin_amdgcn_readfirstlane(pending * ninst));
        waitcnt_lgkm0();  // this wavefront's reads of slot cur are complete
        // every wavefront: stage l + 1 landed, done reading slot cur
        __builtin_amdgcn_s_barrier();
        if constexpr (NCS >= 2) load_frags(nx, 0, 0);  // the last chunk-step uses slot 1
      }
      // last chunk-step; its slots open the window of stage l + ns (into slot cur)
      const bool load2 = OPEN || l + ns < a.kLoop;
      StageBase sb2{0, 0, 0};
      if (load2) sb2 = StageBase{ga2, gb2, cur_b};
#pragma unroll
      for (int q = 0; q < TMTN; ++q) {
        mfma1((NCS - 1) & 1, q);
        dma_at(sb2, load2, q, open);
      }
      if constexpr (NCS == 1) {
        if (more) load_frags(nx, 0, 0);
      }
    };
    int l = 0, cur = 0;
    uint32_t cur_b = static_cast<uint32_t>(lds0);
    // origins of stage ns (as integers: stage ns may lie past the end of K,
    // then only stage ns − 1 = ga2 − stepA is ever loaded from them)
    const uint64_t zA = static_cast<uint64_t>(z) * static_cast<uint64_t>(BK) * 2u;
    uint64_t ga2 = uniform_ptr(Ag) + zA + static_cast<uint64_t>(ns) * stepA;
    uint64_t gb2 = uniform_ptr(Bg) + zA * static_cast<uint64_t>(a.N) + static_cast<uint64_t>(ns) * stepB;
    auto advance = [&]() __attribute__((always_inline)) {
      ++l;
      ga2 += stepA;
      gb2 += stepB;
      if (++cur == ns) {
        cur = 0;
        cur_b = static_cast<uint32_t>(lds0);
      } else {
        cur_b += stage16;
      }
    };
    while (l + ns < a.kLoop) {
      stage_step(l, cur, cur_b, ga2, gb2, std::true_type{});
      advance();
    }
    while (l < a.kLoop) {
      stage_step(l, cur, cur_b, ga2, gb2, std::false_type{});
      advance();
    }
  };
  if (ninst == kMaxDlInst)
    run(std::integral_constant<int, kMaxDlInst>{});
  else if (ninst == kMaxDlInst / 2)
    run(std::integral_constant<int, kMaxDlInst / 2>{});
  else
    run(std::integral_constant<int, 0>{});

  float* Cw = a.C + static_cast<int64_t>(gm) * BM * a.N + static_cast<int64_t>(gn) * BN;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
      for (int e = 0; e < NACC; ++e) {
        const int r = wm * a.WM + i * I + out_row<I>(lane, e);
        const int c = wn * a.WN + j * I + (lane % I);
        put(a.atomic != 0, Cw + static_cast<int64_t>(r) * a.N + c, acc[i][j][e]);
      }
    }
  }
}

// Launch bound: the largest wavefront count the legitimacy rule admits for
// this accumulator size (acc + 96 ≤ 512 / ⌈waves/4⌉); the fast path is used
// with at most 8 wavefronts.
template <int I, int TM, int TN>
constexpr int max_waves() {
  constexpr int acc = TM * TN * I * I / 64;
  return acc + 96 <= 128 ? 16 : (acc + 96 <= 256 ? 8 : 4);
}

template <int I, int TM, int TN, int CPR>
constexpr int launch_threads() {
  return 64 * (CPR > 0 && max_waves<I, TM, TN>() > 8 ? 8 : max_waves<I, TM, TN>());
}

// CPR = 0: generic path; CPR > 0: fast path with BK = CPR·VEC.
template <int DT, int I, int TM, int TN, int CPR>
__global__ void __launch_bounds__((launch_threads<I, TM, TN, CPR>())) gemm_kernel(KArgs a) {
  extern __shared__ u32x4 gt_smem[];
  char* smem = reinterpret_cast<char*>(gt_smem);
  if constexpr (CPR > 0)
    gemm_fast<DT, I, TM, TN, CPR>(a, smem);
  else
    gemm_generic<DT, I, TM, TN>(a, smem);
}

// Register-staged fast path for a K-major A.
template <int DT, int I, int TM, int TN, int CPR>
__global__ void __launch_bounds__((launch_threads<I, TM, TN, CPR>())) gemm_kernel_akm(KArgs a) {
  extern __shared__ u32x4 gt_smem[];
  gemm_fast<DT, I, TM, TN, CPR, true>(a, reinterpret_cast<char*>(gt_smem));
}

// bf16 fast path with direct global→LDS loads: a kernel of its own, so that
// its register allocation does not inherit the register-staged path's.
template <int I, int TM, int TN, int CPR>
__global__ void __launch_bounds__((launch_threads<I, TM, TN, CPR>())) gemm_kernel_dl(KArgs a) {
  extern __shared__ u32x4 gt_smem[];
  gemm_fast_dl<I, TM, TN, CPR>(a, reinterpret_cast<char*>(gt_smem));
}

using LaunchFn = hipError_t (*)(const KArgs&, dim3, dim3, size_t, hipStream_t);

// Raises the kernel's dynamic LDS limit once per device (bit d of `attr_devs`
// for device d < 64; beyond that on every launch), then launches. Concurrent
// callers may both set the attribute, which is idempotent.
template <class F>
hipError_t launch_one(F fn, std::atomic<uint64_t>& attr_devs, const KArgs& a, dim3 grid,
                      dim3 block, size_t lds, hipStream_t s) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev >= 0 && dev < 64 ? uint64_t{1} << dev : 0;
  if (!bit || !(attr_devs.load(std::memory_order_acquire) & bit)) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                            hipFuncAttributeMaxDynamicSharedMemorySize, 163840);
    if (e != hipSuccess) return e;
    attr_devs.fetch_or(bit, std::memory_order_release);
  }
  hipLaunchKernelGGL(fn, grid, block, lds, s, a);
  return hipGetLastError();
}

// AKM: the translation unit instantiates the K-major-A fast path (it then
// serves only launches with a.aKM set; the generic path handles both layouts).
template <int DT, int I, int TM, int TN, int CPR, bool AKM = false>
hipError_t launch_gemm(const KArgs& a, dim3 grid, dim3 block, size_t lds, hipStream_t s) {
  if constexpr (AKM) {
    static_assert(CPR > 0, "the K-major-A kernel is a fast-path kernel");
    static std::atomic<uint64_t> attr_akm{0};
    return launch_one(gemm_kernel_akm<DT, I, TM, TN, CPR>, attr_akm, a, grid, block, lds, s);
  } else {
    if constexpr (DT == 1 && CPR > 0) {
      if (a.dl) {
        static std::atomic<uint64_t> attr_dl{0};
        return launch_one(gemm_kernel_dl<I, TM, TN, CPR>, attr_dl, a, grid, block, lds, s);
      }
    }
    static std::atomic<uint64_t> attr{0};
    return launch_one(gemm_kernel<DT, I, TM, TN, CPR>, attr, a, grid, block, lds, s);
  }
}

// (TM, TN) pairs with TM·TN ≤ 16 (I = 32) and ≤ 64 (I = 16): the register
// rule acc = TM·TN·I²/64 ≤ 256.
#define GT_PAIRS_16(X)                                                                      \
  X(1, 1) X(1, 2) X(2, 1) X(1, 4) X(2, 2) X(4, 1) X(1, 8) X(2, 4) X(4, 2) X(8, 1) X(1, 16) \
      X(2, 8) X(4, 4) X(8, 2) X(16, 1)
#define GT_PAIRS_64(X)                                                                       \
  GT_PAIRS_16(X)                                                                             \
  X(1, 32) X(2, 16) X(4, 8) X(8, 4) X(16, 2) X(32, 1) X(1, 64) X(2, 32) X(4, 16) X(8, 8)     \
      X(16, 4) X(32, 2) X(64, 1)

// Chunks per LDS row with a fast-path instantiation (BK = CPR·VEC).
constexpr int kFastCpr[] = {2, 4, 8, 16};

// Kernel of (dtype, I, CPR, TM, TN), CPR = 0 for the generic path, akm for
// the K-major-A fast path (f32 only); nullptr when not instantiated.
LaunchFn find_gemm_kernel(int dtype, int I, int cpr, int TM, int TN, bool akm);

}  // namespace gt
