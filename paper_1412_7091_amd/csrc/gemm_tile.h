// One output tile of the fp32 MFMA panel GEMM, as a device function shared by
// the step kernel, plus the global-memory helpers of the large-product kernel.
//
// The products of the minibatch algorithm (Appendix A steps 1, 2, 4, 7, 8, 10)
// are small (m = 16 .. 512 on one side, d = 32 .. 1024 on the others), so
// their time goes to memory latency rather than to MFMA throughput.  A tile
// therefore streams K in chunks through a ring of LDS stages that are filled by
// LDS-DMA (global_load_lds): each lane of a wave hands one 16-byte (or 4-byte)
// piece of global memory straight to LDS without passing through registers, so
// the loads of several chunks are in flight while earlier chunks are
// multiplied.  Lanes that fall outside an operand read a block of zeros
// instead, which zero-fills ragged edges without a branch.  Four waves share a
// tile (2 x 2), each owning (T/2)^2 outputs computed with v_mfma_f32_16x16x4f32.
//
// Operands are "virtual" row-major matrices (stacked row blocks, VMat).  In a
// stage an operand whose rows are the output dimension ("KC": k contiguous) is
// stored as T rows of CK floats, and one whose rows are k ("NK") as CK rows of
// T floats.  The 16-byte slots of each row are XOR-swizzled so that the MFMA
// fragment reads of 16 lanes spread over distinct banks; the DMA side applies
// the same swizzle by choosing which global element each lane fetches.
#pragma once

#include "lst_internal.h"

namespace lst {

typedef float floatx4 __attribute__((ext_vector_type(4)));

#ifdef LST_TIMING
// Phase marks of the last GEMM tiles (latency studies only).
static __device__ unsigned long long g_gemm_marks[4][8192][5];
#define LST_MARK(k)                                                              \
  do {                                                                           \
    if (threadIdx.x == 0 && blockIdx.x < 8192)                                   \
      g_gemm_marks[bt.timing_slot & 3][blockIdx.x][k] = wall_clock64();          \
  } while (0)
#else
#define LST_MARK(k) \
  do {              \
  } while (0)
#endif

// ----------------------------------------------- virtual matrices (global)
// Row block of a virtual matrix chosen with constant indices only, so the
// descriptor stays in scalar registers and a lane only selects between them.
__device__ __forceinline__ const float* vm_row(const VMat& v, int row) {
  const float* base = v.p[0];
  int ld = v.ld[0], r0 = 0;
  if (v.nb > 1 && row >= v.r1) { base = v.p[1]; ld = v.ld[1]; r0 = v.r1; }
  return base + (size_t)(row - r0) * (size_t)ld;
}

__device__ __forceinline__ float4 vm_load4(const VMat& v, int row, int col, int nrows, int ncols) {
  float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
  if (row >= nrows || col >= ncols) return o;
  const float* base = vm_row(v, row);
  if (v.vec && col + 3 < ncols) {
    o = *reinterpret_cast<const float4*>(base + col);
  } else {
    o.x = base[col];
    if (col + 1 < ncols) o.y = base[col + 1];
    if (col + 2 < ncols) o.z = base[col + 2];
    if (col + 3 < ncols) o.w = base[col + 3];
  }
  if (v.rscale) {
    const float s = v.rscale[row];
    o.x *= s; o.y *= s; o.z *= s; o.w *= s;
  }
  return o;
}

// ------------------------------------------------------------- LDS-DMA
// 16 bytes of zeros: the source of every DMA lane outside its operand.
static __device__ __attribute__((aligned(16))) float g_dma_zero[4] = {0.f, 0.f, 0.f, 0.f};

__device__ __forceinline__ unsigned lds_u32(const void* p) {
  return (unsigned)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// One LDS-DMA instruction: lane l copies 16 (dma16) or 4 (dma4) bytes from its
// own global address gp to LDS byte address lds + 16 l (4 l); lds must be the
// same for the whole wave.  The compiler does not see these as memory
// operations on LDS, so waits for them are explicit (wait_vm_le) and the
// barrier that publishes them is lds_barrier.  The LDS address travels in m0
// (the compiler itself puts nothing in m0 in these kernels); an SALU write of
// m0 needs one wait state before an LDS-DMA instruction reads it.
__device__ __forceinline__ void dma16(const float* gp, unsigned lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(gp)
               : "memory", "m0");
}
__device__ __forceinline__ void dma4(const float* gp, unsigned lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, off"
               :
               : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(gp)
               : "memory", "m0");
}

// Waits until at most t of this wave's vector-memory operations are
// outstanding, for the largest t <= n on a fixed ladder (waiting for fewer than
// asked is always safe: they complete in issue order).
__device__ __forceinline__ void wait_vm_le(int n) {
  n = __builtin_amdgcn_readfirstlane(n);
  if (n >= 60) asm volatile("s_waitcnt vmcnt(60)" ::: "memory");
  else if (n >= 48) asm volatile("s_waitcnt vmcnt(48)" ::: "memory");
  else if (n >= 32) asm volatile("s_waitcnt vmcnt(32)" ::: "memory");
  else if (n >= 24) asm volatile("s_waitcnt vmcnt(24)" ::: "memory");
  else if (n >= 16) asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
  else if (n >= 12) asm volatile("s_waitcnt vmcnt(12)" ::: "memory");
  else if (n >= 8) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
  else if (n >= 6) asm volatile("s_waitcnt vmcnt(6)" ::: "memory");
  else if (n >= 4) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  else if (n >= 2) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// Workgroup barrier after this wave's LDS writes have landed; also a compiler
// barrier for every memory access.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// ------------------------------------------------------------ the tile
template <int T>
struct PanelGeom {
  static constexpr int CK = 2048 / T;     // k per chunk: 64 (T = 32) or 32 (T = 64)
  static constexpr int OPF = T * CK;      // floats of one operand in a stage
  static constexpr int STAGE = 2 * OPF;   // floats of a stage (A, then B): 16 KB
  static constexpr int WT = T / 2;        // wave tile edge
  static constexpr int IB = WT / 16;      // 16 x 16 blocks per wave tile edge
  static constexpr int KC_SLOTS = CK / 4; // 16-byte slots of a KC row
  static constexpr int NK_SLOTS = T / 4;  // 16-byte slots of an NK row
  static constexpr int DMA16_PER_WAVE = OPF / 256 / 4;  // 16-byte DMA per operand and chunk
  static constexpr int DMA4_PER_WAVE = OPF / 64 / 4;    // 4-byte DMA per operand and chunk
};

constexpr int kPanelStageBytes = 16384;

// Slot swizzles: a KC row r keeps logical slot s at s ^ (r & 7); an NK row k
// at s ^ swz_nk(k), which puts the rows k and k + 4 that two 16-lane groups
// read together into different banks.
template <int T>
__device__ __forceinline__ int swz_nk(int k) {
  return ((k >> 2) & (PanelGeom<T>::NK_SLOTS / 4 - 1)) << 2;
}

// A KC operand's DMA pieces of one lane: the lane copies the same rows and
// the same k offsets within every chunk, so the row pointers are found once.
template <int T, int W>
struct KcPlan {
  static constexpr int NI =
      (W == 4) ? PanelGeom<T>::DMA16_PER_WAVE : PanelGeom<T>::DMA4_PER_WAVE;
  const float* rp[NI];  // row base, or nullptr for a row outside [0, nout)
  int koff[NI];         // k offset of the piece within a chunk (swizzled slot)
};

template <int T, int W>
__device__ __forceinline__ void kc_plan(const VMat& v, int o0, int nout, KcPlan<T, W>& pl) {
  using G = PanelGeom<T>;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int u = 0; u < KcPlan<T, W>::NI; ++u) {
    const int e = 64 * (wave + 4 * u) + lane;
    int row, koff;
    if (W == 4) {  // piece e: 16-byte slot e % KC_SLOTS of stage row e / KC_SLOTS
      row = e / G::KC_SLOTS;
      koff = 4 * ((e % G::KC_SLOTS) ^ (row & 7));
    } else {       // piece e: float e % CK of stage row e / CK
      row = e / G::CK;
      const int pc = e % G::CK;
      koff = 4 * ((pc >> 2) ^ (row & 7)) + (pc & 3);
    }
    const int o = o0 + row;
    pl.rp[u] = o < nout ? vm_row(v, o) : nullptr;
    pl.koff[u] = koff;
  }
}

// Rows [o0, o0 + T) x k in [k0, k0 + CK) of a KC operand (planned by kc_plan)
// into stage region S as S[row][slot ^ (row & 7)].  Elements outside
// [0, nout) x [0, kend) read as zero.  W = 4 needs 16-byte aligned rows and
// kend % 4 == 0.
template <int T, int W>
__device__ __forceinline__ void fill_kc(const KcPlan<T, W>& pl, int k0, int kend, float* S) {
  const int wave = threadIdx.x >> 6;
  const unsigned base = lds_u32(S);
  const float* zero = g_dma_zero;
#pragma unroll
  for (int u = 0; u < KcPlan<T, W>::NI; ++u) {
    const int j = wave + 4 * u;  // instruction j fills stage floats [256 j, +256) (W = 4) or [64 j, +64)
    const int k = k0 + pl.koff[u];
    const float* gp = (pl.rp[u] != nullptr && k < kend) ? pl.rp[u] + k : zero;
    if (W == 4)
      dma16(gp, base + 1024u * j);
    else
      dma4(gp, base + 256u * j);
  }
}

// k in [k0, k0 + CK) x columns [o0, o0 + T) of an NK operand into stage region
// S.  Elements outside [0, kend) x [0, nout) read as zero, except that with
// W = 4 the last 16-byte piece of a row may carry columns >= nout (they only
// reach outputs that are never stored).  W = 4 needs 16-byte aligned rows.
template <int T, int W>
__device__ __forceinline__ void fill_nk(const VMat& v, int o0, int nout, int k0, int kend,
                                        float* S) {
  using G = PanelGeom<T>;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned base = lds_u32(S);
  const float* zero = g_dma_zero;
  if (W == 4) {
#pragma unroll
    for (int u = 0; u < G::DMA16_PER_WAVE; ++u) {
      const int j = wave + 4 * u;
      const int e = 64 * j + lane;
      const int kr = e / G::NK_SLOTS, ps = e % G::NK_SLOTS;
      const int k = k0 + kr, o = o0 + 4 * (ps ^ swz_nk<T>(kr));
      dma16((k < kend && o < nout) ? vm_row(v, k) + o : zero, base + 1024u * j);
    }
  } else {
#pragma unroll
    for (int u = 0; u < G::DMA4_PER_WAVE; ++u) {
      const int j = wave + 4 * u;
      const int e = 64 * j + lane;
      const int kr = e / T, pc = e % T;
      const int k = k0 + kr, o = o0 + 4 * ((pc >> 2) ^ swz_nk<T>(kr)) + (pc & 3);
      dma4((k < kend && o < nout) ? vm_row(v, k) + o : zero, base + 256u * j);
    }
  }
}

// MFMA operand fragments of one 16-wide k slice: MFMA q of the slice pairs
// k = kk + 4 g + q of A and of B (g = lane / 16), so a lane holds 4 values
// of row/column l16 per 16 x 16 block.
template <int T, int AKC, int BKC>
__device__ __forceinline__ void load_frags(const float* As, const float* Bs, int kk,
                                           float (&a)[PanelGeom<T>::IB][4],
                                           float (&b)[PanelGeom<T>::IB][4]) {
  using G = PanelGeom<T>;
  constexpr int IB = G::IB;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int g = lane >> 4, l16 = lane & 15;
#pragma unroll
  for (int i = 0; i < IB; ++i) {
    const int r = wm * G::WT + i * 16 + l16;
    if (AKC) {
      const int slot = (kk >> 2) + g;
      const float4 f = *reinterpret_cast<const float4*>(As + r * G::CK + 4 * (slot ^ (r & 7)));
      a[i][0] = f.x; a[i][1] = f.y; a[i][2] = f.z; a[i][3] = f.w;
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int k = kk + 4 * g + q;
        a[i][q] = As[k * T + 4 * ((r >> 2) ^ swz_nk<T>(k)) + (r & 3)];
      }
    }
  }
#pragma unroll
  for (int j = 0; j < IB; ++j) {
    const int c = wn * G::WT + j * 16 + l16;
    if (BKC) {
      const int slot = (kk >> 2) + g;
      const float4 f = *reinterpret_cast<const float4*>(Bs + c * G::CK + 4 * (slot ^ (c & 7)));
      b[j][0] = f.x; b[j][1] = f.y; b[j][2] = f.z; b[j][3] = f.w;
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int k = kk + 4 * g + q;
        b[j][q] = Bs[k * T + 4 * ((c >> 2) ^ swz_nk<T>(k)) + (c & 3)];
      }
    }
  }
}

// Accumulators of a wave: with one 16 x 16 block per wave (T = 32) the four
// MFMAs of a slice alternate between two accumulator sets so that no MFMA
// waits for the result of the one just before it; the sets are added at the end.
template <int T>
struct Accum {
  static constexpr int IB = PanelGeom<T>::IB;
  static constexpr int NS = IB == 1 ? 2 : 1;
  floatx4 v[NS][IB][IB];
};

template <int T>
__device__ __forceinline__ void mma_frags(const float (&a)[PanelGeom<T>::IB][4],
                                          const float (&b)[PanelGeom<T>::IB][4], Accum<T>& acc) {
  constexpr int IB = PanelGeom<T>::IB, NS = Accum<T>::NS;
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int i = 0; i < IB; ++i)
#pragma unroll
      for (int j = 0; j < IB; ++j)
        acc.v[q % NS][i][j] =
            __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][q], b[j][q], acc.v[q % NS][i][j], 0, 0, 0);
}

// acc += the first nsl 16-wide k slices held in consecutive stages from
// smem (slice s lives in stage s / (CK / 16)).  The fragments of slice s + 1
// are read from LDS while the MFMAs of slice s run.
// 32-tiles with both operands k-contiguous (the stacked product of the first
// launch, the m x m products): the fragment reads go through inline asm, one
// slice ahead of the MFMAs they feed, and each slice waits only for the pair
// of reads issued a slice earlier.  Left to the compiler, the wait for a
// slice's fragments lands right after the reads of the next slice were issued
// (it counts outstanding LDS reads conservatively across the loop), so every
// slice pays the LDS latency.  The per-lane offsets of the four slices of a
// stage are computed once.  Slices past nsl inside the last stage are read
// (inside the stage) but not multiplied.
__device__ __forceinline__ void lds_read_pair(floatx4& a, floatx4& b, unsigned pa, unsigned pb) {
  asm volatile("ds_read_b128 %0, %2\n\tds_read_b128 %1, %3" : "=&v"(a), "=&v"(b) : "v"(pa), "v"(pb));
}
// Waits until at most the pair issued after (a, b) is outstanding.
__device__ __forceinline__ void lds_wait_pair(floatx4& a, floatx4& b) {
  asm volatile("s_waitcnt lgkmcnt(2)" : "+v"(a), "+v"(b));
}

__device__ __forceinline__ void mma_pair32(const floatx4& a, const floatx4& b, Accum<32>& acc) {
  acc.v[0][0][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b.x, acc.v[0][0][0], 0, 0, 0);
  acc.v[1][0][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b.y, acc.v[1][0][0], 0, 0, 0);
  acc.v[0][0][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b.z, acc.v[0][0][0], 0, 0, 0);
  acc.v[1][0][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b.w, acc.v[1][0][0], 0, 0, 0);
}

__device__ __forceinline__ void mma_slices_kc32(const float* smem, int nsl, Accum<32>& acc) {
  using G = PanelGeom<32>;
  constexpr unsigned SB = G::STAGE * 4;  // bytes per stage
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, l16 = lane & 15;
  const int ra = (wave >> 1) * G::WT + l16, rb = (wave & 1) * G::WT + l16;
  const unsigned base = lds_u32(smem);
  unsigned oa[4], ob[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    oa[j] = base + 4u * (unsigned)(ra * G::CK + 4 * ((4 * j + g) ^ (ra & 7)));
    ob[j] = base + 4u * (unsigned)(G::OPF + rb * G::CK + 4 * ((4 * j + g) ^ (rb & 7)));
  }
  if (nsl <= 0) return;
  const int nst = (nsl + 3) >> 2;
  floatx4 a0, b0, a1, b1;
  lds_read_pair(a0, b0, oa[0], ob[0]);
  for (int st = 0; st < nst; ++st) {
    const unsigned sb = (unsigned)st * SB, nb = (st + 1 < nst) ? sb + SB : sb;
    const int s0 = 4 * st;
    lds_read_pair(a1, b1, oa[1] + sb, ob[1] + sb);
    lds_wait_pair(a0, b0);
    mma_pair32(a0, b0, acc);  // slice s0 < nsl always
    lds_read_pair(a0, b0, oa[2] + sb, ob[2] + sb);
    lds_wait_pair(a1, b1);
    if (s0 + 1 < nsl) mma_pair32(a1, b1, acc);
    lds_read_pair(a1, b1, oa[3] + sb, ob[3] + sb);
    lds_wait_pair(a0, b0);
    if (s0 + 2 < nsl) mma_pair32(a0, b0, acc);
    lds_read_pair(a0, b0, oa[0] + nb, ob[0] + nb);
    lds_wait_pair(a1, b1);
    if (s0 + 3 < nsl) mma_pair32(a1, b1, acc);
  }
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a0), "+v"(b0));
}

template <int T, int AKC, int BKC>
__device__ __forceinline__ void mma_slices(const float* smem, int nsl, Accum<T>& acc) {
  if constexpr (T == 32 && AKC && BKC) {
    mma_slices_kc32(smem, nsl, acc);
    return;
  }
  using G = PanelGeom<T>;
  constexpr int IB = G::IB, NKK = G::CK / 16;
  auto frags = [&](int sl, float (&a)[IB][4], float (&b)[IB][4]) {
    const float* st = smem + (sl / NKK) * G::STAGE;
    load_frags<T, AKC, BKC>(st, st + G::OPF, (sl % NKK) * 16, a, b);
  };
  float a0[IB][4], b0[IB][4], a1[IB][4], b1[IB][4];
  if (nsl <= 0) return;
  // The prefetch index is clamped rather than guarded, so the reads carry no
  // branch and the compiler can wait for exactly the fragments it uses.
  frags(0, a0, b0);
  for (int sl = 0; sl < nsl; sl += 2) {
    frags(min(sl + 1, nsl - 1), a1, b1);
    mma_frags<T>(a0, b0, acc);
    if (sl + 1 >= nsl) break;
    frags(min(sl + 2, nsl - 1), a0, b0);
    mma_frags<T>(a1, b1, acc);
  }
}

// Operand layouts a kernel instantiation supports (bit masks).
enum : unsigned { V_NT = 2, V_NN = 4, V_TN = 8 };

// Epilogue-mask bit (beyond the Epi values) of the per-row partial sums that
// EPI_STORE can produce (GemmProblem::dotp, GemmProblem::absp); kernels
// without it compile neither.
constexpr unsigned EPX_ROWSUMS = 8;
// Epilogue-mask bit of kernels whose GEMM blocks test the batch's skip_if flag
// only before their epilogue (they read their operands either way): the
// flag's load, which needs the descriptor's pointer first, then overlaps the
// operand fetch instead of preceding it.  Without it the caller tests the
// flag before the tile starts.
constexpr unsigned EPX_LATE_SKIP = 9;

// P.epi == e, folded away when the instantiation does not support e.
template <unsigned EPIS>
__device__ __forceinline__ bool epi_is(const GemmProblem& P, int e) {
  return ((EPIS >> e) & 1u) && P.epi == e;
}

// The tile (tm, tn) of problem P over k in [kb, ke) with bt.stages stages in
// smem, then its epilogue (one of the epilogues in the mask EPIS).
template <int T, int W, int AKC, int BKC, unsigned EPIS>
__device__ __forceinline__ void panel_run(const GemmBatch& bt, const GemmProblem& P, int tm,
                                          int tn, int z, int kb, int ke, float* smem) {
  using G = PanelGeom<T>;
  constexpr int IB = G::IB;
  const int S = bt.stages;
  const int m0 = tm * T, n0 = tn * T;
  const GemmExtras& X = bt.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  constexpr bool kRowSums = (EPIS >> EPX_ROWSUMS) & 1u;
  constexpr bool kLateSkip = (EPIS >> EPX_LATE_SKIP) & 1u;
  const int skip = (kLateSkip && bt.skip_if != nullptr) ? *bt.skip_if : 0;
  const bool dot = kRowSums && X.dotp != nullptr && n0 < X.dot_ncols;
  const bool absr = kRowSums && X.absp != nullptr && n0 + T > X.abs_col0;
  LST_MARK(0);

  // Operands of the epilogue, fetched before the first chunk.
  float pre1[IB][IB][4], pre2[IB][IB][4];
#pragma unroll
  for (int i = 0; i < IB; ++i)
#pragma unroll
    for (int j = 0; j < IB; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm * G::WT + i * 16 + 4 * (lane >> 4) + r;
        const int col = n0 + wn * G::WT + j * 16 + (lane & 15);
        pre1[i][j][r] = 0.f;
        pre2[i][j][r] = 0.f;
        if (row >= P.M || col >= P.N) continue;
        if (((epi_is<EPIS>(P, EPI_STORE) || epi_is<EPIS>(P, EPI_SCALED)) && P.beta != 0.f) ||
            (epi_is<EPIS>(P, EPI_SYM) && row <= col && P.beta != 0.f)) {
          pre1[i][j][r] = P.C[(size_t)row * P.ldc + col];
        } else if (epi_is<EPIS>(P, EPI_GRADN)) {
          pre1[i][j][r] = X.s1[row] * X.e1[(size_t)row * X.lde1 + col] +
                          X.s2[row] * X.e2[(size_t)row * X.lde2 + col];
        } else if (epi_is<EPIS>(P, EPI_GRADT)) {
          // accumulator rows 2o and 2o + 1 (r even / odd) both feed output row o
          const int o = row >> 1;
          if ((r & 1) == 0) {
            pre1[i][j][r] = X.s1[o] * X.e1[(size_t)o * X.lde1 + col];
            pre2[i][j][r] = X.s2[o] * X.e2[(size_t)o * X.lde2 + col];
          } else {
            pre1[i][j][r] = X.s1[o];
            pre2[i][j][r] = X.s2[o];
          }
        }
        if (dot && col < X.dot_ncols) pre2[i][j][r] = X.dot_h[(size_t)row * X.ld_doth + col];
      }

  Accum<T> acs;
#pragma unroll
  for (int u = 0; u < Accum<T>::NS; ++u)
#pragma unroll
    for (int i = 0; i < IB; ++i)
#pragma unroll
      for (int j = 0; j < IB; ++j) acs.v[u][i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int nch = ke > kb ? (ke - kb + G::CK - 1) / G::CK : 0;
  constexpr int NI = (W == 4) ? G::DMA16_PER_WAVE : G::DMA4_PER_WAVE;
  const int I = 2 * NI;  // DMA instructions per wave and chunk
  KcPlan<T, W> pa, pb;
  if (AKC) kc_plan<T, W>(P.A, m0, P.M, pa);
  if (BKC) kc_plan<T, W>(P.B, n0, P.N, pb);
  auto fill = [&](int c) {
    float* st = smem + (c % S) * G::STAGE;
    const int k0 = kb + c * G::CK;
    if (AKC)
      fill_kc<T, W>(pa, k0, ke, st);
    else
      fill_nk<T, W>(P.A, m0, P.M, k0, ke, st);
    if (BKC)
      fill_kc<T, W>(pb, k0, ke, st + G::OPF);
    else
      fill_nk<T, W>(P.B, n0, P.N, k0, ke, st + G::OPF);
  };
  // Every chunk fits (chunk c in stage c): all are issued at once.  Otherwise
  // a ring keeps S - 1 chunks ahead of the one being multiplied.
  const bool resident = nch <= S;
  const int ahead = resident ? nch : S - 1;
  for (int c = 0; c < ahead; ++c) fill(c);
  LST_MARK(1);
  if (resident) {
    // one wait, then one uninterrupted MFMA loop over all of K
    wait_vm_le(0);
    lds_barrier();
    LST_MARK(2);
    mma_slices<T, AKC, BKC>(smem, (ke - kb + 15) / 16, acs);
  } else {
    for (int c = 0; c < nch; ++c) {
      // chunks issued so far: min(nch, c + S - 1); wait for chunk c only
      const int issued = (c + S - 1 < nch) ? c + S - 1 : nch;
      wait_vm_le((issued - c - 1) * I);
      lds_barrier();
      if (c == 0) LST_MARK(2);
      if (c + S - 1 < nch) fill(c + S - 1);  // reuses the stage of chunk c - 1
      const int kc = ke - (kb + c * G::CK);
      mma_slices<T, AKC, BKC>(smem + (c % S) * G::STAGE,
                              kc >= G::CK ? G::CK / 16 : (kc + 15) / 16, acs);
    }
  }
  floatx4 acc[IB][IB];
#pragma unroll
  for (int i = 0; i < IB; ++i)
#pragma unroll
    for (int j = 0; j < IB; ++j) {
      acc[i][j] = acs.v[0][i][j];
      if (Accum<T>::NS == 2) acc[i][j] += acs.v[Accum<T>::NS - 1][i][j];
    }

  // The epilogue's operands were fetched before the K loop.  Waiting for them
  // here, once, keeps the waits out of the stores below: the compiler would
  // otherwise wait at each element's first use, and on this chip those waits
  // also wait for every store issued before them.
#pragma unroll
  for (int i = 0; i < IB; ++i)
#pragma unroll
    for (int j = 0; j < IB; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) asm volatile("" ::"v"(pre1[i][j][r]), "v"(pre2[i][j][r]));

  LST_MARK(3);
  if (kLateSkip && skip != 0) return;  // nothing is written
  // EPI_SCALED: the power-of-two scale from the trace of the previous product
  // (exact, so the vector the products converge to does not depend on it).
  float pscale = 1.f, tsum = 0.f;
  if (epi_is<EPIS>(P, EPI_SCALED) && X.s1 != nullptr) {
    const float t = *X.s1;
    if (t > 0.f && isfinite(t)) pscale = ldexpf(1.f, max(-126, min(126, -2 * ilogbf(t))));
  }
  // Element r of acc[i][j]: row 4*(lane/16) + r, column lane % 16 of its 16 x 16 block.
  float dsum[IB][4], asum[IB][4];
#pragma unroll
  for (int i = 0; i < IB; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) dsum[i][r] = asum[i][r] = 0.f;
#pragma unroll
  for (int i = 0; i < IB; ++i)
#pragma unroll
    for (int j = 0; j < IB; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm * G::WT + i * 16 + 4 * (lane >> 4) + r;
        const int col = n0 + wn * G::WT + j * 16 + (lane & 15);
        if (row >= P.M || col >= P.N) continue;
        const float v = acc[i][j][r];
        if (epi_is<EPIS>(P, EPI_STORE)) {
          P.C[(size_t)row * P.ldc + col] = P.alpha * v + P.beta * pre1[i][j][r];
          if (dot && col < X.dot_ncols) dsum[i][r] += pre2[i][j][r] * v;
          if (absr && col >= X.abs_col0) asum[i][r] += fabsf(v);
        } else if (epi_is<EPIS>(P, EPI_SYM)) {
          if (row <= col) {
            const float o = pre1[i][j][r] + P.alpha * v;
            P.C[(size_t)row * P.ldc + col] = o;
            P.C[(size_t)col * P.ldc + row] = o;
          }
        } else if (epi_is<EPIS>(P, EPI_GRADT)) {
          if ((r & 1) == 0) {  // row is even; row + 1 sits in element r + 1 of this lane
            const int o = row >> 1;
            const float gv = pre1[i][j][r] + pre2[i][j][r];
            const float nh = pre1[i][j][r + 1] * v + pre2[i][j][r + 1] * acc[i][j][r + 1];
            X.g[(size_t)o * X.ldg + col] = gv;
            P.C[(size_t)o * P.ldc + col] = gv + P.alpha * nh;
          }
        } else if (epi_is<EPIS>(P, EPI_GRADN)) {
          X.g[(size_t)row * X.ldg + col] = pre1[i][j][r];
          P.C[(size_t)row * P.ldc + col] = pre1[i][j][r] + P.alpha * v;
        } else if (epi_is<EPIS>(P, EPI_STORE_T)) {
          const float o = P.alpha * v;
          P.C[(size_t)row * P.ldc + col] = o;
          P.C[(size_t)P.ct_off + (size_t)col * P.ldc + row] = o;
        } else if (epi_is<EPIS>(P, EPI_PARTIAL)) {
          P.C[(size_t)z * P.M * P.N + (size_t)row * P.N + col] = v;
        } else if (epi_is<EPIS>(P, EPI_SCALED)) {
          const float o = P.alpha * pscale * v + P.beta * pre1[i][j][r];
          P.C[(size_t)row * P.ldc + col] = o;
          if (row == col) tsum += o;
        }
      }
  if (epi_is<EPIS>(P, EPI_SCALED) && X.g != nullptr && tm == tn) {
    // the diagonal of a tile on the diagonal: one atomic per wave
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) tsum += __shfl_xor(tsum, off);
    if (lane == 0) atomicAdd(X.g, tsum);
  }
  if (dot) {
    // Row sums over this wave's columns, reduced across the 16 lanes of a row
    // in a fixed butterfly; one partial per (row, tile column, wave column).
#pragma unroll
    for (int i = 0; i < IB; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float v = dsum[i][r];
        v += __shfl_xor(v, 1);
        v += __shfl_xor(v, 2);
        v += __shfl_xor(v, 4);
        v += __shfl_xor(v, 8);
        const int row = m0 + wm * G::WT + i * 16 + 4 * (lane >> 4) + r;
        if ((lane & 15) == 0 && row < P.M) X.dotp[(size_t)row * X.ld_dotp + 2 * tn + wn] = v;
      }
  }
  if (absr) {  // the same for the sums of |C| (a wave left of abs_col0 writes 0)
    const int pc = 2 * (tn - X.abs_col0 / T) + wn;
#pragma unroll
    for (int i = 0; i < IB; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float v = asum[i][r];
        v += __shfl_xor(v, 1);
        v += __shfl_xor(v, 2);
        v += __shfl_xor(v, 4);
        v += __shfl_xor(v, 8);
        const int row = m0 + wm * G::WT + i * 16 + 4 * (lane >> 4) + r;
        if ((lane & 15) == 0 && row < P.M) X.absp[(size_t)row * X.ld_absp + pc] = v;
      }
  }
  LST_MARK(4);
}

// Workgroups are dispatched to the 8 XCDs round-robin (block b to XCD b % 8),
// each XCD with its own L2.  Block b gets tile xcd_tile(b): every XCD takes
// one contiguous run of the tile sequence, so tiles that read the same
// operand panels share an L2.  A bijection of [0, total).
__device__ __forceinline__ int xcd_tile(int b, int total) {
  const int x = b & 7, li = b >> 3;
  const int q = total >> 3, r = total & 7;
  return x * q + min(x, r) + li;
}

// The operand layouts of problem P (one of VARS) for tile edge T.
template <int T, int W, unsigned VARS, unsigned EPIS>
__device__ __forceinline__ void panel_layout(const GemmBatch& bt, const GemmProblem& P, int tm,
                                             int tn, int z, int kb, int ke, float* smem) {
  if ((VARS & V_NT) && P.a_kc && P.b_kc)
    panel_run<T, W, 1, 1, EPIS>(bt, P, tm, tn, z, kb, ke, smem);
  else if ((VARS & V_NN) && P.a_kc && !P.b_kc)
    panel_run<T, W, 1, 0, EPIS>(bt, P, tm, tn, z, kb, ke, smem);
  else if ((VARS & V_TN) && !P.a_kc)
    panel_run<T, W, 0, 0, EPIS>(bt, P, tm, tn, z, kb, ke, smem);
}

// Tile-edge masks of a kernel instantiation.
enum : unsigned { TILE32 = 1, TILE64 = 2 };

// Computes the tile of block t of the batch (problems laid out one after
// another, each in column-panel-major order); smem holds bt.stages stages of
// kPanelStageBytes.  Only the tile edges in TILES, the layouts in VARS and the
// epilogues in EPIS are compiled (the host checks every problem).
template <unsigned TILES, int W, unsigned VARS, unsigned EPIS>
__device__ __forceinline__ void panel_tile(const GemmBatch& bt, int t, float* smem) {
  t = xcd_tile(t, bt.total_tiles);
  int q = 0;
  while (q + 1 < bt.np && t >= bt.tile_begins[q + 1]) ++q;
  if (bt.skip_updates_if && q >= bt.first_update && *bt.skip_updates_if) return;
  // A private copy: the inline-asm memory clobbers of the pipeline would
  // otherwise make every use re-read the descriptor from kernel arguments.
  const GemmProblem P = bt.p[q];
  int lt = t - P.tile_begin;
  int tm, tn, kb = 0, ke = P.K, z = 0;
  if (epi_is<EPIS>(P, EPI_SYM)) {
    int TT = P.tiles_m, r = 0;
    while (lt >= TT - r) { lt -= TT - r; ++r; }
    tm = r; tn = r + lt;
  } else {
    const int per = P.tiles_m * P.tiles_n;
    z = lt / per;
    lt -= z * per;
    tn = lt / P.tiles_m;  // the tiles of one B panel are consecutive
    tm = lt - tn * P.tiles_m;
    if (P.ksplit > 1) {
      const int kc = ((P.K + P.ksplit - 1) / P.ksplit + 15) / 16 * 16;
      kb = z * kc;
      ke = min(P.K, kb + kc);
    }
  }
  if ((TILES & TILE64) && P.tile == 64)
    panel_layout<64, W, VARS, EPIS>(bt, P, tm, tn, z, kb, ke, smem);
  else if (TILES & TILE32)
    panel_layout<32, W, VARS, EPIS>(bt, P, tm, tn, z, kb, ke, smem);
}

// Layout bit of a problem (matches the dispatch above).
__host__ __device__ inline unsigned problem_variant(const GemmProblem& P) {
  if (P.a_kc && P.b_kc) return V_NT;
  if (P.a_kc) return V_NN;
  return V_TN;
}

}  // namespace lst
