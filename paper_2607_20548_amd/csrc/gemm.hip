// fp32 GEMM on the CDNA4 matrix cores (v_mfma_f32_32x32x2_f32), used for every
// dense product of the SOAP step: the factor EMAs (one triangle), the power
// products L Q_L and R Q_R, the rotations and the compact-WY updates of the QR.
//
// Tiling: a 256-thread workgroup (4 wave64s in a 2 x 2 arrangement) computes a
// 128 x 128 tile of C; each wave owns a 64 x 64 sub-tile held as 2 x 2 MFMA
// 32x32 accumulators (64 accumulation registers per lane).  K advances in slabs
// of 16 staged through double-buffered LDS; the global loads run two slabs
// ahead in two register sets (also for the rank-k updates, whose few slabs
// would otherwise each wait for their loads), with every load issued
// unconditionally at a clamped address so that the waits cover exactly the
// slab being stored.  Both operands are kept in LDS as
// [x][k] rows (x = output row or column, k contiguous, padded to 20 floats so
// that 16-byte reads of 16 consecutive lanes fall in distinct banks); a lane
// then fetches the 8 k-values it feeds to 8 consecutive MFMAs with two
// ds_read_b128.  Within a 16-slab, lane half h of the MFMA operand carries
// k = 8h + s at MFMA step s; A and B use the same assignment, so the sum over
// k is complete.
//
// Epilogue: the tile goes through LDS (free after the K loop) so that C is read
// and written 16 bytes per lane (see the epilogue).
//
// Tile order: the 8 XCDs receive workgroups round-robin, so the linear tile
// index is remapped to give each XCD a contiguous run of tiles, and that run is
// walked in groups of 8 tile-rows so that neighbouring tiles share A rows and B
// columns in the XCD's L2.
#include "internal.h"

namespace soap {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int BK = 16;
constexpr int LDSK = BK + 4;            // padded LDS row stride in floats ([x][k] rows)
constexpr int TILE_FLOATS = 128 * LDSK;  // one operand tile in LDS
// [k][x] rows of an x-contiguous operand (vector path): 128 x-values padded to
// 132 floats, so that the two lane halves of a fragment read (k and k + 8)
// fall in disjoint banks.
constexpr int LDSX = BN + 4;
static_assert(BK * LDSX <= TILE_FLOATS, "an x-contiguous slab must fit one tile buffer");
constexpr int NTHREADS = 256;
constexpr int SHORT_K = 512;    // products with at most this much K per slice use the rank-k kernel
constexpr int GROUP_M = 8;


enum { MODE_GENERAL = 0, MODE_SYRK = 1, MODE_ADAM = 2 };

struct KParams {
  int M, N, K;
  const float *A;
  int64_t lda, sA;
  const float *B;
  int64_t ldb, sB;
  float *C;
  int64_t ldc, sC;
  float alpha, beta;
  float *V;
  float *Nout;
  float b2, c1, c2, eps;
  int tiles_m, tiles_n, ntiles;
  int kslice;       // K extent of one split-K slice (multiple of BK); = K when not split
  float *part;      // split-K partials, or nullptr
  const unsigned *skip;   // batch entry b is skipped when skip[b * sSkip] != 0 (or nullptr)
  int64_t sSkip;
};

// Loads one operand slab of 128 x-rows by BK k-values into registers.
//   KCONTIG = true : global element (x, k) at base[x*ld + k]
//   KCONTIG = false: global element (x, k) at base[k*ld + x]
// Work split: 512 (x, k-quad) items over 256 threads, two per thread; with
// VEC == 4 an x-contiguous slab is instead read either as 4 x 2 blocks
// (k-quad, x pair; 8-byte loads), one per thread, transposed in registers to
// [x][k] rows, or (KX) as 512 (k, x-quad) items with 16-byte loads, each wave
// covering two k rows per load instruction, kept in LDS as [k][x] rows
// exactly as loaded.  The rank-k kernel takes the second form (5-7% faster
// at K = 128-512: the register copies of the transposition had made its
// loads wait right after their issue); for the long-K kernel it measured 1%
// slower (its fragments then need eight 4-byte LDS reads instead of two
// 16-byte ones).
template <bool KCONTIG, int VEC, bool KX = false>
struct SlabLoader {
  float r[8];

  // Every load is issued unconditionally at an address clamped into the
  // matrix: with no branch around the loads the compiler can wait for exactly
  // the loads a store needs, which the two-slab prefetch of the long-K loop
  // relies on.  With VEC == 4 the values are used as loaded: rows x >= X only
  // reach output rows or columns that are never written, and k-values past
  // the end of K are zeroed by store() (kvalid), right before they go to LDS,
  // so that nothing consumes a loaded register early.  The scalar path
  // (VEC == 1) masks both at load time.  Requires X >= 1, K >= 1 (and the
  // VEC == 4 preconditions: K % 4 == 0 for k-contiguous, X even for
  // x-contiguous operands, and with KX X % 4 == 0 and a leading dimension
  // and base aligned to 16 bytes).
  __device__ __forceinline__ void load(const float *__restrict__ base, int64_t ld, int x0,
                                       int k0, int X, int K, int tid) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int idx = tid + NTHREADS * s;
      if (KCONTIG) {
        const int x = x0 + (idx >> 2);
        const int k = k0 + 4 * (idx & 3);
        const int64_t row = (int64_t)min(x, X - 1) * ld;
        if (VEC == 4) {
          const float4 v = *reinterpret_cast<const float4 *>(base + row + min(k, K - 4));
          r[4 * s + 0] = v.x; r[4 * s + 1] = v.y; r[4 * s + 2] = v.z; r[4 * s + 3] = v.w;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float v = base[row + min(k + e, K - 1)];
            r[4 * s + e] = (x < X && k + e < K) ? v : 0.f;
          }
        }
      } else if (VEC == 4 && KX) {
        // x-contiguous with 16-byte loads: wave w reads k rows 8s + 2w (lanes
        // 0-31) and 8s + 2w + 1 (lanes 32-63), four consecutive x per lane.
        // The row address is formed on the scalar unit (k is uniform within
        // each half wave; the second half adds one row, or none at the end
        // of K), each lane adds its column offset.
        const int lane = tid & 63;
        const int kb = k0 + 8 * s + 2 * __builtin_amdgcn_readfirstlane(tid >> 6);
        const float *rowp = base + (int64_t)min(kb, K - 1) * ld;
        const int64_t dr = (kb < K - 1) ? ld : 0;
        const unsigned xc = (unsigned)min(x0 + 4 * (lane & 31), X - 4);
        const float4 v = *reinterpret_cast<const float4 *>(rowp + ((lane >> 5) ? dr : 0) + xc);
        r[4 * s + 0] = v.x; r[4 * s + 1] = v.y; r[4 * s + 2] = v.z; r[4 * s + 3] = v.w;
      } else if (VEC == 4) {
        // x-contiguous with 8-byte loads: thread -> (k-quad, x pair); the
        // 4 x 2 block is transposed in registers (r[0..3] = column x,
        // r[4..7] = column x+1).  Needs an even x extent and leading
        // dimension.  k is uniform within a wave, so the row address is
        // formed on the scalar unit and each lane adds its column offset.
        if (s == 0) {
          const int x = x0 + 2 * (tid & 63);
          const int k = k0 + 4 * __builtin_amdgcn_readfirstlane(tid >> 6);
          const unsigned xc = (unsigned)min(x, X - 2);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float *rowp = base + (int64_t)min(k + e, K - 1) * ld;
            const float2 v = *reinterpret_cast<const float2 *>(rowp + xc);
            r[e] = v.x;
            r[4 + e] = v.y;
          }
        }
      } else {
        const int x = x0 + (idx & 127);
        const int k = k0 + 4 * (idx >> 7);
        const int xc = min(x, X - 1);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float v = base[(int64_t)min(k + e, K - 1) * ld + xc];
          r[4 * s + e] = (x < X && k + e < K) ? v : 0.f;
        }
      }
    }
  }

  // Writes the slab to LDS, as [x][k] rows ([k][x] rows for an x-contiguous
  // operand on the vector path); kvalid = number of k-values of this slab
  // inside K (BK except in the last, ragged slab).
  __device__ __forceinline__ void store(float *lds, int tid, int kvalid) {
    if (!KCONTIG && VEC == 4 && KX) {
      const int lane = tid & 63, w = tid >> 6;
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int k = 8 * s + 2 * w + (lane >> 5);
        float4 v = make_float4(r[4 * s + 0], r[4 * s + 1], r[4 * s + 2], r[4 * s + 3]);
        if (k >= kvalid) v = make_float4(0.f, 0.f, 0.f, 0.f);
        *reinterpret_cast<float4 *>(lds + k * LDSX + 4 * (lane & 31)) = v;
      }
      return;
    }
    if (VEC == 4 && kvalid < BK) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int idx = tid + NTHREADS * s;
        const int kl = KCONTIG ? 4 * (idx & 3) : 4 * (tid >> 6);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (KCONTIG) {
            if (kl >= kvalid) r[4 * s + e] = 0.f;   // K % 4 == 0: whole quads
          } else if (s == 0 && kl + e >= kvalid) {
            r[e] = 0.f;
            r[4 + e] = 0.f;
          }
        }
      }
    }
    if (!KCONTIG && VEC == 4) {
      const int xl = 2 * (tid & 63), kq = tid >> 6;
      *reinterpret_cast<float4 *>(lds + xl * LDSK + 4 * kq) = make_float4(r[0], r[1], r[2], r[3]);
      *reinterpret_cast<float4 *>(lds + (xl + 1) * LDSK + 4 * kq) =
          make_float4(r[4], r[5], r[6], r[7]);
      return;
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int idx = tid + NTHREADS * s;
      const int x = KCONTIG ? (idx >> 2) : (idx & 127);
      const int kq = KCONTIG ? (idx & 3) : (idx >> 7);
      *reinterpret_cast<float4 *>(lds + x * LDSK + 4 * kq) =
          make_float4(r[4 * s + 0], r[4 * s + 1], r[4 * s + 2], r[4 * s + 3]);
    }
  }
};

// The 8 k-values k = 8h + s (s = 0..7) of operand row x from LDS: two 16-byte
// reads from [x][k] rows, or (KX) eight 4-byte reads from [k][x] rows.
template <bool KX>
__device__ __forceinline__ void read_frag(const float *lds, int x, int h, float (&f)[8]) {
  if constexpr (KX) {
#pragma unroll
    for (int s = 0; s < 8; ++s) f[s] = lds[(8 * h + s) * LDSX + x];
  } else {
    const float4 lo = *reinterpret_cast<const float4 *>(lds + x * LDSK + 8 * h);
    const float4 hi = *reinterpret_cast<const float4 *>(lds + x * LDSK + 8 * h + 4);
    f[0] = lo.x; f[1] = lo.y; f[2] = lo.z; f[3] = lo.w;
    f[4] = hi.x; f[5] = hi.y; f[6] = hi.z; f[7] = hi.w;
  }
}

// Maps the linear workgroup id to a (tile-row, tile-column) pair.
template <int MODE>
__device__ __forceinline__ void tile_coords(const KParams &p, int t, int &tm, int &tn) {
  const int nt = p.ntiles;
  if ((nt & 7) == 0) t = (t & 7) * (nt >> 3) + (t >> 3);  // contiguous run per XCD
  if (MODE == MODE_SYRK) {
    // lower-triangle tiles (tm >= tn), enumerated row by row
    int r = (int)((sqrtf(8.f * (float)t + 1.f) - 1.f) * 0.5f);
    while ((r + 1) * (r + 2) / 2 <= t) ++r;
    while (r * (r + 1) / 2 > t) --r;
    tm = r;
    tn = t - r * (r + 1) / 2;
  } else {
    const int per_group = GROUP_M * p.tiles_n;
    const int group = t / per_group;
    const int first_m = group * GROUP_M;
    const int gsz = min(p.tiles_m - first_m, GROUP_M);
    const int in_group = t - group * per_group;
    tm = first_m + in_group % gsz;
    tn = in_group / gsz;
  }
}

// MINB > 1 marks the short-K variant (K per slice <= SHORT_K, the QR's
// rank-k updates): the bound on resident workgroups makes the compiler keep
// the accumulators in VGPRs (4 workgroups per CU), and the epilogue batches
// its reads of C.  Long-K products (MINB = 1) keep the accumulators in AGPRs.
template <int TA, int TB, int VEC, int MODE, int TAG, int MINB, bool PERSIST = false>
__global__ __launch_bounds__(NTHREADS, MINB) void gemm_f32_mfma(KParams p) {
  constexpr bool SHORTK = MINB > 1;
  __shared__ __attribute__((aligned(16))) float lds[2 * 2 * TILE_FLOATS];
  if (p.skip && p.skip[(int64_t)blockIdx.z * p.sSkip] != 0u) return;

  // One tile per workgroup; PERSIST: a loop over tiles when the grid was
  // capped (the caller limited the compute units this product may hold).
  for (int tile = blockIdx.x;;) {
  int tm, tn;
  tile_coords<MODE>(p, tile, tm, tn);
  const int64_t bz = blockIdx.z;
  const float *A = p.A + bz * p.sA;
  const float *B = p.B + bz * p.sB;
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int xl = lane & 31, h = lane >> 5;

  // op(A) rows are x = i: k-contiguous when TA == 0.  op(B) columns are x = j:
  // k-contiguous when TB == 1.
  // the rank-k kernel keeps x-contiguous operands as [k][x] rows in LDS
  constexpr bool KXL = SHORTK && VEC == 4;
  SlabLoader<TA == 0, VEC, KXL> la;
  SlabLoader<TB == 1, VEC, KXL> lb;

  v16f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto buf = [&](int stage, int which) { return lds + (stage * 2 + which) * TILE_FLOATS; };

  const int kbeg = blockIdx.y * p.kslice;
  const int kend = min(p.K, kbeg + p.kslice);
  const int nk = (kend - kbeg + BK - 1) / BK;
  // One K slab from LDS buffer `cur` into the accumulators.
  constexpr bool AKX = KXL && TA == 1, BKX = KXL && TB == 0;
  auto compute = [&](int cur) {
    float fa[2][8], fb[2][8];
    read_frag<BKX>(buf(cur, 1), wn * 64 + xl, h, fb[0]);
    read_frag<BKX>(buf(cur, 1), wn * 64 + 32 + xl, h, fb[1]);
    read_frag<AKX>(buf(cur, 0), wm * 64 + xl, h, fa[0]);
    read_frag<AKX>(buf(cur, 0), wm * 64 + 32 + xl, h, fa[1]);
#pragma unroll
    for (int s = 0; s < 8; ++s)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[i][s], fb[j][s], acc[i][j], 0, 0, 0);
  };

  {
    // Global loads run two slabs ahead of the matrix cores (two register
    // sets), so a slab's loads have two slabs of MFMA work to land.
    SlabLoader<TA == 0, VEC, KXL> lc;
    SlabLoader<TB == 1, VEC, KXL> ld;
    auto load_set = [&](SlabLoader<TA == 0, VEC, KXL> &xa, SlabLoader<TB == 1, VEC, KXL> &xb, int kt) {
      const int k0 = kbeg + kt * BK;
      xa.load(A, p.lda, m0, k0, p.M, kend, tid);
      xb.load(B, p.ldb, n0, k0, p.N, kend, tid);
    };
    auto store_set = [&](SlabLoader<TA == 0, VEC, KXL> &xa, SlabLoader<TB == 1, VEC, KXL> &xb, int stage,
                         int kt) {
      const int kvalid = min(BK, kend - (kbeg + kt * BK));
      xa.store(buf(stage, 0), tid, kvalid);
      xb.store(buf(stage, 1), tid, kvalid);
    };
    // slab kt is computed from LDS while the register set `held` carries
    // slab kt+1 (stored to the other buffer after the MFMAs) and `next`
    // receives slab kt+2.
    auto body = [&](int kt, SlabLoader<TA == 0, VEC, KXL> &ha, SlabLoader<TB == 1, VEC, KXL> &hb,
                    SlabLoader<TA == 0, VEC, KXL> &na, SlabLoader<TB == 1, VEC, KXL> &nb) {
      const int cur = kt & 1;
      load_set(na, nb, kt + 2);   // past the end: clamped loads, all zero
      compute(cur);
      if (kt + 1 < nk) store_set(ha, hb, cur ^ 1, kt + 1);
      __syncthreads();
    };
    if (nk > 0) {
      load_set(lc, ld, 0);
      store_set(lc, ld, 0, 0);
      load_set(la, lb, 1);
    }
    __syncthreads();
    for (int kt = 0; kt < nk; kt += 2) {
      body(kt, la, lb, lc, ld);
      if (kt + 1 < nk) body(kt + 1, lc, ld, la, lb);
    }
  }

  // Epilogue.  Accumulator register r of block (i, j) holds
  // C[row0 + 8*(r/4) + 4*h + r%4][col0 + xl].
  float *C = p.C + bz * p.sC;
  float *P = p.part ? p.part + (bz * gridDim.y + blockIdx.y) * (int64_t)p.M * p.N : nullptr;
  float *V = (MODE == MODE_ADAM) ? p.V + bz * p.sC : nullptr;
  float *Nout = (MODE == MODE_ADAM) ? p.Nout + bz * p.sC : nullptr;
  // Short-K products (rank-k updates) spend a large share of their time
  // here, so their C values are loaded 16 at a time before any store (the
  // compiler cannot move a load of C above a store to C, and reading one
  // element after storing the previous one serializes 64 memory latencies).
  // Long-K products keep the register-lean element-by-element form.
  bool staged = false;
  if constexpr (MODE == MODE_SYRK && !SHORTK) {
   if ((reinterpret_cast<uintptr_t>(C) & 15u) == 0 && (p.ldc & 3) == 0) {
    staged = true;
    // One triangle, mirrored, through LDS in two halves of 64 rows: the
    // lower part (row >= col) is written as beta C + alpha acc with 16-byte
    // reads and writes, the final values go back to LDS, and the mirror is
    // written from the transposed half, again 16 bytes per lane (scattered
    // 4-byte mirror stores, and a read of C after each store, otherwise).
    constexpr int SLD = BN + 4;
    float *stage = lds;
    const bool read_back = p.beta != 0.f;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      __syncthreads();
      if (wm == half) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              stage[(i * 32 + 8 * (r >> 2) + 4 * h + (r & 3)) * SLD + wn * 64 + j * 32 + xl] =
                  acc[i][j][r];
      }
      __syncthreads();
#pragma unroll
      for (int g4 = 0; g4 < 2; ++g4) {   // two groups of 4 (registers of the main loop)
        float4 cv[4];
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
          const int q = 4 * g4 + qq;
          const int e = tid + NTHREADS * q, lrow = e >> 5, c4 = (e & 31) * 4;
          const int row = m0 + half * 64 + lrow, col = n0 + c4;
          cv[qq] = make_float4(0.f, 0.f, 0.f, 0.f);
          // only the lower triangle is read (a float4 with col <= row holds at
          // least one element of it; the others are masked)
          if (read_back && row < p.M && col <= row && col < p.N) {
            const float *src = C + (int64_t)row * p.ldc + col;
            if (col + 3 < p.N && col + 3 <= row) {
              cv[qq] = *reinterpret_cast<const float4 *>(src);
            } else {
              cv[qq].x = src[0];
              if (col + 1 < p.N && col + 1 <= row) cv[qq].y = src[1];
              if (col + 2 < p.N && col + 2 <= row) cv[qq].z = src[2];
              if (col + 3 < p.N && col + 3 <= row) cv[qq].w = src[3];
            }
          }
        }
        asm volatile("" ::: "memory");
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
          const int q = 4 * g4 + qq;
          const int e = tid + NTHREADS * q, lrow = e >> 5, c4 = (e & 31) * 4;
          const int row = m0 + half * 64 + lrow, col = n0 + c4;
          float *sp = stage + lrow * SLD + c4;
          const float4 a = *reinterpret_cast<const float4 *>(sp);
          float4 v;
          v.x = p.alpha * a.x + (read_back ? p.beta * cv[qq].x : 0.f);
          v.y = p.alpha * a.y + (read_back ? p.beta * cv[qq].y : 0.f);
          v.z = p.alpha * a.z + (read_back ? p.beta * cv[qq].z : 0.f);
          v.w = p.alpha * a.w + (read_back ? p.beta * cv[qq].w : 0.f);
          *reinterpret_cast<float4 *>(sp) = v;   // final values for the mirror
          if (row >= p.M || col > row || col >= p.N) continue;
          float *dst = C + (int64_t)row * p.ldc + col;
          if (col + 3 < p.N && col + 3 <= row) {
            *reinterpret_cast<float4 *>(dst) = v;
          } else {
            dst[0] = v.x;
            if (col + 1 < p.N && col + 1 <= row) dst[1] = v.y;
            if (col + 2 < p.N && col + 2 <= row) dst[2] = v.z;
            if (col + 3 < p.N && col + 3 <= row) dst[3] = v.w;
          }
        }
        asm volatile("" ::: "memory");
      }
      __syncthreads();
      // mirror: C[col][row] for row > col; thread -> (lc = output row within
      // the tile's columns, 4 consecutive rows of this half as output columns)
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int e = tid + NTHREADS * q, lc = e >> 4, r4 = (e & 15) * 4;
        const int orow = n0 + lc, ocol = m0 + half * 64 + r4;   // C[orow][ocol] = value(ocol, orow)
        if (orow >= p.N || ocol >= p.M) continue;
        float4 v;
        v.x = stage[(r4 + 0) * SLD + lc];
        v.y = stage[(r4 + 1) * SLD + lc];
        v.z = stage[(r4 + 2) * SLD + lc];
        v.w = stage[(r4 + 3) * SLD + lc];
        float *dst = C + (int64_t)orow * p.ldc + ocol;
        // element (ocol + u, orow) of the lower triangle mirrors to here when ocol + u > orow
        if (ocol > orow && ocol + 3 < p.M) {
          *reinterpret_cast<float4 *>(dst) = v;
        } else {
          if (ocol > orow) dst[0] = v.x;
          if (ocol + 1 > orow && ocol + 1 < p.M) dst[1] = v.y;
          if (ocol + 2 > orow && ocol + 2 < p.M) dst[2] = v.z;
          if (ocol + 3 > orow && ocol + 3 < p.M) dst[3] = v.w;
        }
      }
    }
    if constexpr (PERSIST) __syncthreads();
   }
  }
  if constexpr (MODE == MODE_GENERAL) {
   if (!P && (reinterpret_cast<uintptr_t>(C) & 15u) == 0 && (p.ldc & 3) == 0) {
    staged = true;
    // Rank-k updates are bound by their pass over C, so the tile goes
    // through LDS (free after the K loop) in two halves of 64 rows and C is
    // read and written 16 bytes per lane, all reads of a thread before its
    // stores.
    constexpr int SLD = BN + 4;   // padded LDS row (64 rows x 132 floats fit the 40 KB)
    float *stage = lds;
    const bool read_back = p.beta != 0.f;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      __syncthreads();
      if (wm == half) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              stage[(i * 32 + 8 * (r >> 2) + 4 * h + (r & 3)) * SLD + wn * 64 + j * 32 + xl] =
                  acc[i][j][r];
      }
      __syncthreads();
      float4 cv[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int e = tid + NTHREADS * q, lrow = e >> 5, c4 = (e & 31) * 4;
        const int row = m0 + half * 64 + lrow, col = n0 + c4;
        cv[q] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (read_back && row < p.M) {
          const float *src = C + (int64_t)row * p.ldc + col;
          if (col + 3 < p.N) {
            cv[q] = *reinterpret_cast<const float4 *>(src);
          } else {
            if (col < p.N) cv[q].x = src[0];
            if (col + 1 < p.N) cv[q].y = src[1];
            if (col + 2 < p.N) cv[q].z = src[2];
          }
        }
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int e = tid + NTHREADS * q, lrow = e >> 5, c4 = (e & 31) * 4;
        const int row = m0 + half * 64 + lrow, col = n0 + c4;
        if (row >= p.M) continue;
        const float4 a = *reinterpret_cast<const float4 *>(stage + lrow * SLD + c4);
        float4 v;
        v.x = p.alpha * a.x + (read_back ? p.beta * cv[q].x : 0.f);
        v.y = p.alpha * a.y + (read_back ? p.beta * cv[q].y : 0.f);
        v.z = p.alpha * a.z + (read_back ? p.beta * cv[q].z : 0.f);
        v.w = p.alpha * a.w + (read_back ? p.beta * cv[q].w : 0.f);
        float *dst = C + (int64_t)row * p.ldc + col;
        if (col + 3 < p.N) {
          *reinterpret_cast<float4 *>(dst) = v;
        } else {
          if (col < p.N) dst[0] = v.x;
          if (col + 1 < p.N) dst[1] = v.y;
          if (col + 2 < p.N) dst[2] = v.z;
        }
      }
    }
    // a persistent launch's next tile writes the same LDS
    if constexpr (PERSIST) __syncthreads();
   }
  }
  if (staged) {
    // done
  } else if constexpr (SHORTK) {
   {
    const bool read_back = !P && p.beta != 0.f;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int col = n0 + wn * 64 + j * 32 + xl;
        float cv[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
          const int64_t off = (int64_t)row * p.ldc + col;
          cv[r] = 0.f;
          if (read_back && row < p.M && col < p.N) cv[r] = C[off];
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
          if (row >= p.M || col >= p.N) continue;
          const int64_t off = (int64_t)row * p.ldc + col;
          if (P) {
            P[(int64_t)row * p.N + col] = acc[i][j][r];
          } else {
            float v = p.alpha * acc[i][j][r];
            if (p.beta != 0.f) v += p.beta * cv[r];
            C[off] = v;
          }
        }
      }
   }
  } else {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int col = n0 + wn * 64 + j * 32 + xl;
        // C = alpha acc + beta C: the 16 values of C of this block are read
        // before its stores (one memory latency per block instead of one per
        // element); the empty asm keeps the compiler from hoisting the reads
        // of later blocks, whose registers would cost the main loop a wave
        // per SIMD.
        float cv[16];
        if (MODE == MODE_GENERAL && !P) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
            cv[r] = (p.beta != 0.f && row < p.M && col < p.N) ? C[(int64_t)row * p.ldc + col] : 0.f;
          }
        }
        asm volatile("" ::: "memory");
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
          if (row >= p.M || col >= p.N) continue;
          const int64_t off = (int64_t)row * p.ldc + col;
          if (MODE == MODE_GENERAL && P) {
            P[(int64_t)row * p.N + col] = acc[i][j][r];
          } else if (MODE == MODE_GENERAL) {
            float v = p.alpha * acc[i][j][r];
            if (p.beta != 0.f) v += p.beta * cv[r];
            C[off] = v;
          } else if (MODE == MODE_SYRK) {
            if (row < col) continue;  // the mirror of (col,row) is written by its owner
            const float v = (p.beta != 0.f ? p.beta * C[off] : 0.f) + p.alpha * acc[i][j][r];
            C[off] = v;
            if (row != col) C[(int64_t)col * p.ldc + row] = v;
          } else if ((r & 1) == 0) {
            // rows 2i, 2i+1 of the interleaved operand are G' and M' of
            // output row i; they sit in registers r, r+1 of the same lane
            const float g = acc[i][j][r];
            const float mm = acc[i][j][r + 1];
            const int64_t o = (int64_t)(row >> 1) * p.ldc + col;
            const float v = p.b2 * V[o] + (1.f - p.b2) * g * g;
            V[o] = v;
            Nout[o] = (mm / p.c1) / (sqrtf(v / p.c2) + p.eps);
          }
        }
      }
  }
  if constexpr (!PERSIST) break;
  tile += gridDim.x;
  if (tile >= p.ntiles) break;
  }  // tile loop
}

// C = alpha * sum_s part[s] + beta * C, slices summed in index order.
__global__ __launch_bounds__(256) void splitk_reduce(const float *__restrict__ part, int S,
                                                     int M, int N, float *C, int64_t ldc,
                                                     int64_t sC, float alpha, float beta,
                                                     const unsigned *skip, int64_t sSkip) {
  const int64_t bz = blockIdx.y;
  if (skip && skip[bz * sSkip] != 0u) return;
  const int64_t mn = (int64_t)M * N;
  const float *pb = part + bz * S * mn;
  float *Cb = C + bz * sC;
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < mn; e += (int64_t)gridDim.x * 256) {
    float acc = 0.f;
    for (int s = 0; s < S; ++s) acc += pb[s * mn + e];
    const int64_t row = e / N, col = e - row * N;
    float v = alpha * acc;
    if (beta != 0.f) v += beta * Cb[row * ldc + col];
    Cb[row * ldc + col] = v;
  }
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// vec_ok, vec_ok_kx: the vector path's preconditions for the long-K kernel
// and for the rank-k kernel (vec_ok_for).
template <int MODE>
hipError_t dispatch(const GemmDesc &d, KParams &kp, hipStream_t s, bool vec_ok, bool vec_ok_kx) {
  dim3 block(NTHREADS);
  const int S = (MODE == MODE_GENERAL && d.splitk > 1 && d.part) ? d.splitk : 1;
  // A cap counts every workgroup (split slices and batch included); the
  // tile dimension stays a multiple of 8 for XCD locality.
  const int64_t per_tile = (int64_t)S * d.batch;
  const bool capped = (MODE == MODE_GENERAL || MODE == MODE_SYRK) && d.max_wg > 0 &&
                      (int64_t)kp.ntiles * per_tile > d.max_wg;
  const int wgs = capped ? (int)std::max<int64_t>(8, (d.max_wg / per_tile) & ~int64_t(7)) : kp.ntiles;
  dim3 grid(std::min(wgs, kp.ntiles), S, (unsigned)d.batch);
#define SOAP_LAUNCH(TA, TB, VEC, TAG) \
  hipLaunchKernelGGL((gemm_f32_mfma<TA, TB, VEC, MODE, TAG, 1>), grid, block, 0, s, kp)
  const int code = d.trans_a * 2 + d.trans_b;
  if (MODE == MODE_SYRK && capped) {
    // the two layouts of the factor products: X X^T (0, 1) and X^T X (1, 0)
#define SOAP_LAUNCH_SP(TA, TB, VEC) \
  hipLaunchKernelGGL((gemm_f32_mfma<TA, TB, VEC, MODE_SYRK, 0, 1, true>), grid, block, 0, s, kp)
    if (code == 1) { if (vec_ok) SOAP_LAUNCH_SP(0, 1, 4); else SOAP_LAUNCH_SP(0, 1, 1); }
    else if (code == 2) { if (vec_ok) SOAP_LAUNCH_SP(1, 0, 4); else SOAP_LAUNCH_SP(1, 0, 1); }
    else return hipErrorInvalidValue;
#undef SOAP_LAUNCH_SP
  } else if (capped) {
#define SOAP_LAUNCH_P(TA, TB, VEC, MINB) \
  hipLaunchKernelGGL((gemm_f32_mfma<TA, TB, VEC, MODE_GENERAL, 0, MINB, true>), grid, block, 0, s, kp)
    const bool shortk = kp.kslice <= SHORT_K;
    switch (code * 4 + ((shortk ? vec_ok_kx : vec_ok) ? 2 : 0) + (shortk ? 1 : 0)) {
      case 0: SOAP_LAUNCH_P(0, 0, 1, 1); break;
      case 1: SOAP_LAUNCH_P(0, 0, 1, 3); break;
      case 2: SOAP_LAUNCH_P(0, 0, 4, 1); break;
      case 3: SOAP_LAUNCH_P(0, 0, 4, 3); break;
      case 4: SOAP_LAUNCH_P(0, 1, 1, 1); break;
      case 5: SOAP_LAUNCH_P(0, 1, 1, 3); break;
      case 6: SOAP_LAUNCH_P(0, 1, 4, 1); break;
      case 7: SOAP_LAUNCH_P(0, 1, 4, 3); break;
      case 8: SOAP_LAUNCH_P(1, 0, 1, 1); break;
      case 9: SOAP_LAUNCH_P(1, 0, 1, 3); break;
      case 10: SOAP_LAUNCH_P(1, 0, 4, 1); break;
      case 11: SOAP_LAUNCH_P(1, 0, 4, 3); break;
      case 12: SOAP_LAUNCH_P(1, 1, 1, 1); break;
      case 13: SOAP_LAUNCH_P(1, 1, 1, 3); break;
      case 14: SOAP_LAUNCH_P(1, 1, 4, 1); break;
      default: SOAP_LAUNCH_P(1, 1, 4, 3); break;
    }
#undef SOAP_LAUNCH_P
  } else if (MODE == MODE_GENERAL && d.tag != 0 && code == 2) {
    // the power products (transposed-A layout) under their own symbols
    if (d.tag == 1) { if (vec_ok) SOAP_LAUNCH(1, 0, 4, 1); else SOAP_LAUNCH(1, 0, 1, 1); }
    else { if (vec_ok) SOAP_LAUNCH(1, 0, 4, 2); else SOAP_LAUNCH(1, 0, 1, 2); }
  } else if (MODE == MODE_GENERAL && kp.kslice <= SHORT_K) {
#define SOAP_LAUNCH_RANK(TA, TB, VEC) \
  hipLaunchKernelGGL((gemm_f32_mfma<TA, TB, VEC, MODE_GENERAL, 0, 3>), grid, block, 0, s, kp)
    if (vec_ok_kx) {
      switch (code) {
        case 0: SOAP_LAUNCH_RANK(0, 0, 4); break;
        case 1: SOAP_LAUNCH_RANK(0, 1, 4); break;
        case 2: SOAP_LAUNCH_RANK(1, 0, 4); break;
        default: SOAP_LAUNCH_RANK(1, 1, 4); break;
      }
    } else {
      switch (code) {
        case 0: SOAP_LAUNCH_RANK(0, 0, 1); break;
        case 1: SOAP_LAUNCH_RANK(0, 1, 1); break;
        case 2: SOAP_LAUNCH_RANK(1, 0, 1); break;
        default: SOAP_LAUNCH_RANK(1, 1, 1); break;
      }
    }
#undef SOAP_LAUNCH_RANK
  } else if (vec_ok) {
    switch (code) {
      case 0: SOAP_LAUNCH(0, 0, 4, 0); break;
      case 1: SOAP_LAUNCH(0, 1, 4, 0); break;
      case 2: SOAP_LAUNCH(1, 0, 4, 0); break;
      default: SOAP_LAUNCH(1, 1, 4, 0); break;
    }
  } else {
    switch (code) {
      case 0: SOAP_LAUNCH(0, 0, 1, 0); break;
      case 1: SOAP_LAUNCH(0, 1, 1, 0); break;
      case 2: SOAP_LAUNCH(1, 0, 1, 0); break;
      default: SOAP_LAUNCH(1, 1, 1, 0); break;
    }
  }
#undef SOAP_LAUNCH
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || S == 1 || d.partials_only) return err;
  int64_t mn = d.M * d.N;
  unsigned gx = (unsigned)std::min<int64_t>((mn + 255) / 256, 2048);
  hipLaunchKernelGGL(splitk_reduce, dim3(gx, (unsigned)d.batch), dim3(256), 0, s, kp.part, S,
                     kp.M, kp.N, d.C, d.ldc, d.sC, d.alpha, d.beta, kp.skip, kp.sSkip);
  return hipGetLastError();
}

KParams make_params(const GemmDesc &d) {
  KParams kp{};
  kp.M = (int)d.M; kp.N = (int)d.N; kp.K = (int)d.K;
  kp.A = d.A; kp.lda = d.lda; kp.sA = d.sA;
  kp.B = d.B; kp.ldb = d.ldb; kp.sB = d.sB;
  kp.C = d.C; kp.ldc = d.ldc; kp.sC = d.sC;
  kp.alpha = d.alpha; kp.beta = d.beta;
  kp.tiles_m = (int)((d.M + BM - 1) / BM);
  kp.tiles_n = (int)((d.N + BN - 1) / BN);
  kp.ntiles = kp.tiles_m * kp.tiles_n;
  kp.kslice = (int)d.K;
  kp.part = nullptr;
  kp.skip = d.skip;
  kp.sSkip = d.sSkip;
  if (d.splitk > 1 && d.part) {
    const int64_t per = (d.K + d.splitk - 1) / d.splitk;
    kp.kslice = (int)(((per + BK - 1) / BK) * BK);
    kp.part = d.part;
  }
  return kp;
}

// Vector loads: a k-contiguous operand uses 16-byte loads along k (k extent,
// leading dimension, batch stride multiples of 4 floats, 16-byte aligned
// base); an x-contiguous operand uses 8-byte loads along x (even x extent,
// leading dimension and batch stride, 8-byte aligned base).

bool aligned8(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 7u) == 0; }

// The vector path's preconditions; kx: the rank-k kernel, whose x-contiguous
// operands are read 16 bytes at a time along x.
bool vec_ok_for(const GemmDesc &d, bool kx) {
  bool ok = true;
  if (d.trans_a == 0)
    ok = ok && d.K % 4 == 0 && d.lda % 4 == 0 && d.sA % 4 == 0 && aligned16(d.A);
  else if (kx)
    ok = ok && d.M % 4 == 0 && d.lda % 4 == 0 && d.sA % 4 == 0 && aligned16(d.A);
  else
    ok = ok && d.M % 2 == 0 && d.lda % 2 == 0 && d.sA % 2 == 0 && aligned8(d.A);
  if (d.trans_b == 1)
    ok = ok && d.K % 4 == 0 && d.ldb % 4 == 0 && d.sB % 4 == 0 && aligned16(d.B);
  else if (kx)
    ok = ok && d.N % 4 == 0 && d.ldb % 4 == 0 && d.sB % 4 == 0 && aligned16(d.B);
  else
    ok = ok && d.N % 2 == 0 && d.ldb % 2 == 0 && d.sB % 2 == 0 && aligned8(d.B);
  return ok;
}

}  // namespace

int choose_splitk(int64_t M, int64_t N, int64_t K, int64_t batch, int max_split) {
  const int64_t tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN) * batch;
  if (tiles <= 0) return 1;   // an empty product: nothing to split
  int64_t s = (512 + tiles - 1) / tiles;
  const int64_t kcap = K / 512;     // keep at least 512 of K per slice
  if (s > kcap) s = kcap;
  if (s > max_split) s = max_split;
  if (s < 1) s = 1;
  return (int)s;
}

hipError_t launch_gemm(const GemmDesc &d, hipStream_t s) {
  if (d.M <= 0 || d.N <= 0 || d.batch <= 0) return hipSuccess;
  KParams kp = make_params(d);
  return dispatch<MODE_GENERAL>(d, kp, s, vec_ok_for(d, false), vec_ok_for(d, true));
}

hipError_t launch_syrk_ema(const GemmDesc &d, hipStream_t s) {
  if (d.M <= 0 || d.batch <= 0) return hipSuccess;
  KParams kp = make_params(d);
  kp.ntiles = kp.tiles_m * (kp.tiles_m + 1) / 2;
  return dispatch<MODE_SYRK>(d, kp, s, vec_ok_for(d, false), vec_ok_for(d, true));
}

hipError_t launch_gemm_adam(const GemmDesc &d, const AdamEpi &e, hipStream_t s) {
  if (d.M <= 0 || d.N <= 0 || d.batch <= 0) return hipSuccess;
  if (d.M % 2 != 0 || d.trans_a != 0) return hipErrorInvalidValue;
  KParams kp = make_params(d);
  kp.V = e.V;
  kp.Nout = e.Nout;
  kp.b2 = e.b2; kp.c1 = e.c1; kp.c2 = e.c2; kp.eps = e.eps;
  return dispatch<MODE_ADAM>(d, kp, s, vec_ok_for(d, false), vec_ok_for(d, true));
}

}  // namespace soap
