// Weight gradient of a 3x3, stride-1, padding-1 convolution on gfx950 MFMA, staged by
// pixel patches:
//   dW[o][(r, s, c)] = sum over pixels (n, p, q) of dy[n][p][q][o] * x[n][p + r - 1][q + s - 1][c],
// and the same kernel's 1x1 form (KH = 1: dW[o][c] = sum over pixels of dy[.][o] x[.][c],
// steps of 64 consecutive pixels, no halo, chunks of up to 288 input channels).
//
// A block owns one tile of output channels (64 or 96 rows) by one chunk of input channels
// (32, or 48 for inputs whose channel count is a multiple of 48 but not of 32) across all
// nine taps, and walks a contiguous range of PR x PC pixel patches of one image each.  Per
// patch it stages in LDS, once, the patch's dy pixels and the (PR + 2) x (PC + 2) input
// pixels that the nine taps reach (zeros outside the image), and reads every tap's MFMA
// operand out of that halo with transposing LDS reads at the tap's pixel shift.  The
// general weight-gradient kernel gathers each tap's input rows for every 128-column tile,
// so its load path carries each input element nine times and dy once per column tile;
// here an input element crosses it about 1.4 times per output-channel tile and dy once per
// channel chunk, about a quarter of the bytes per FLOP.
//
// Eight waves in two halves.  Each half holds the whole tile's accumulators (the tile's
// 32 x 32 MFMA blocks dealt to its four waves in contiguous runs of at most seven), and
// the halves take alternate 16-pixel slices of every patch.  At the end the halves add
// their sums through LDS and the block writes one fp32 partial (dW itself for a single
// split; accumulate honoured there).  Every sum runs in a fixed pixel order, so the
// result is bitwise reproducible.
//
// Loads write LDS directly (buffer_load ... lds; lane i of a wave instruction deposits its
// 16 bytes at the instruction's LDS base + 16 i), every step issues the same number of
// them per wave (loads past the split or outside the image read zeros, and the slots past
// the stage's data fill an unread tail of the stage), and a step waits for exactly its
// own loads.  Each stage is its own LDS object and every load targets the stage it fills,
// so the compiler's load-wait bookkeeping tells the stage being read from the stages
// being filled.
#include <cstdlib>
#include <type_traits>

#include "kernels.h"

namespace numbat {

namespace {

template <int V>
using IcH = std::integral_constant<int, V>;

template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(IcH<I>{});
    static_for<I + 1, N>(f);
  }
}

typedef short hv4s_t __attribute__((ext_vector_type(4)));
typedef unsigned hv2u_t __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void hlds_void_t;
typedef __attribute__((address_space(3))) hv4s_t hlds_v4s_t;
typedef __attribute__((address_space(3))) f32x4 hlds_f4_t;

constexpr uint32_t kOobH = 0x80000000u;  // an offset past every buffer range: the load returns zeros
constexpr int kRecH = 0x7ffffff0;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t hrsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, kRecH, 0x00020000);
}

__device__ __forceinline__ uint32_t lds_u32(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// Tile geometry.  OB: 32-row output-channel blocks (tile of 32 OB channels); CK: input
// channels per chunk; PR x PC: the pixel patch of one step (1 x 64 for the 1x1 form); S:
// LDS stages; KH: kernel side (3, or 1).
template <int OB, int CK, int PR, int PC, int S, int KH>
struct WhShape {
  static constexpr int NP = PR * PC;                // pixels per step
  static constexpr int KS = NP / 16;                // 16-pixel MFMA slices per step
  static constexpr int RB = OB * 64;                // bytes per staged dy pixel
  // bytes per staged input pixel: CK channels; in the 1x1 form padded so that four
  // consecutive pixels start in distinct quarters of the 256-byte bank window
  static constexpr int HRB0 = CK * 2;
  static constexpr int HRB = KH == 3 ? HRB0 : HRB0 % 256 == 128 ? HRB0 + 64 : HRB0 % 256 == 32 ? HRB0 + 32 : HRB0;
  static constexpr int HW = PC + KH - 1, HP = (PR + KH - 1) * HW;  // halo width, halo pixels
  static constexpr int NCOL = KH * KH * CK;         // columns (tap, channel)
  static constexpr int CB = (NCOL + 31) / 32;       // 32-column blocks
  static constexpr int T = OB * CB;                 // 32 x 32 blocks of the tile
  static constexpr int R = (T + 3) / 4;             // blocks per wave
  static constexpr int NCB = (OB + R - 2) / OB + 1; // column blocks one wave's run touches
  static constexpr int NDY = NP * RB / 1024;        // 1 KiB load instructions per stage: dy ...
  static constexpr int NHA = (HP * HRB + 1023) / 1024;  // ... and the halo
  static constexpr int LW = (NDY + NHA + 7) / 8;    // load instructions per wave per step
  static constexpr int STAGE = 8 * LW * 1024;       // bytes per stage (every wave's load slots)
  static constexpr int PENDING = (S - 2) * LW;      // loads of the later stages in flight at a step's wait
  static constexpr int EPS = STAGE / 4096;          // accumulator blocks of a wave one stage holds
  static_assert(KH == 3 ? (NP % 16 == 0 && (PC == 4 || PC == 8 || PC == 16)) : (KH == 1 && PR == 1 && NP % 16 == 0),
                "patch");
  static_assert(NP * RB % 1024 == 0, "dy stage in whole load instructions");
  static_assert(RB == 128 || RB == 192, "dy row");
  static_assert(KH == 3 ? (CK == 32 || CK == 48) : (CK % 16 == 0 && HRB % 16 == 0), "channel chunk");
  static_assert(R <= 7, "accumulator registers");
  static_assert(S >= 3 && S <= 6 && S * EPS >= 4 * R, "stages (they also hold the halves' exchange)");
  static_assert(S * STAGE <= 160 * 1024, "LDS");
  static_assert(PENDING <= 63, "load counter");
};

template <int OB, int CK, int PR, int PC, int S, int KH>
__global__ __launch_bounds__(512) void wgrad_halo_kernel(WgradArgs a, WhGeom g) {
  using Sh = WhShape<OB, CK, PR, PC, S, KH>;
  constexpr int KS = Sh::KS, RB = Sh::RB, HRB = Sh::HRB, HW = Sh::HW, R = Sh::R, NCB = Sh::NCB;
  constexpr int LW = Sh::LW, NDY = Sh::NDY, NHA = Sh::NHA, T = Sh::T, CB = Sh::CB;

  __shared__ __attribute__((aligned(16))) unsigned char sS0[Sh::STAGE];
  __shared__ __attribute__((aligned(16))) unsigned char sS1[Sh::STAGE];
  __shared__ __attribute__((aligned(16))) unsigned char sS2[Sh::STAGE];
  __shared__ __attribute__((aligned(16))) unsigned char sS3[S > 3 ? Sh::STAGE : 16];
  __shared__ __attribute__((aligned(16))) unsigned char sS4[S > 4 ? Sh::STAGE : 16];
  __shared__ __attribute__((aligned(16))) unsigned char sS5[S > 5 ? Sh::STAGE : 16];
  auto stage = [&](auto sc) __attribute__((always_inline)) -> unsigned char* {
    constexpr int s = decltype(sc)::value;
    if constexpr (s == 0) return sS0;
    else if constexpr (s == 1) return sS1;
    else if constexpr (s == 2) return sS2;
    else if constexpr (s == 3) return sS3;
    else if constexpr (s == 4) return sS4;
    else return sS5;
  };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = wave >> 2, wq = wave & 3;
  const uint32_t gx = gridDim.x, gy = gridDim.y;
  const uint32_t lin = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
  const uint32_t lg = a.remap ? xcd_remap(lin, gx * gy * gridDim.z) : lin;
  const int bx = (int)(lg % gx), by = (int)((lg / gx) % gy), bz = (int)(lg / (gx * gy));
  const int o0 = bx * 32 * OB, c0 = by * CK;
  const int pbeg = bz * g.pps;
  const int pend = pbeg + g.pps < g.npatch ? pbeg + g.pps : g.npatch;
  const int nsteps = pend > pbeg ? pend - pbeg : 0;

  // This lane's part of load slot u of its wave (instruction n = wave + 8 u of a stage):
  // the byte offset of its 16 bytes from the step's base (kOobH: zeros) and the position of
  // its pixel: for a halo pixel (row + 1) | (column + 1) << 16 relative to the patch origin
  // (the dy pixels of a patch are always inside); in the 1x1 form the pixel's index within
  // the step (the last step may pass the last pixel).
  uint32_t loff[LW];
  uint32_t lpos[LW];
#pragma unroll
  for (int u = 0; u < LW; ++u) {
    const int n = wave + 8 * u;
    const int bl = n * 1024 + 16 * lane;
    loff[u] = kOobH;
    lpos[u] = KH == 3 ? (1u | (1u << 16)) : 0u;
    if (n < NDY) {
      const int pr = bl / RB, slot = (bl % RB) / 16;
      const int ch = RB == 128 ? (slot ^ (4 * ((pr >> 1) & 1))) : slot;  // 16-byte chunk (8 channels)
      const int o = o0 + 8 * ch;
      if (o < a.co) loff[u] = (uint32_t)(((pr / PC) * a.w + pr % PC) * (uint32_t)a.dy_pix * 2u + (uint32_t)o * 2u);
      if constexpr (KH == 1) lpos[u] = (uint32_t)pr;
    } else if (n < NDY + NHA) {
      const int hb = bl - NDY * 1024;
      const int hp = hb / HRB, ch = (hb % HRB) / 16;
      const int hr = hp / HW, hc = hp % HW;
      const int c = c0 + 8 * ch;
      if (hp < Sh::HP && 8 * ch < CK && c < a.ci)
        loff[u] = (uint32_t)((hr * a.w + hc) * (uint32_t)a.x_pix * 2u + (uint32_t)c * 2u);
      lpos[u] = KH == 3 ? ((uint32_t)hr | ((uint32_t)hc << 16)) : (uint32_t)hp;
    }
  }

  // issue the loads of step st (patch pbeg + st) into stage sc
  auto issue = [&](auto sc, int st) __attribute__((always_inline)) {
    unsigned char* Sg = stage(sc);
    const bool live = st < nsteps;
    int img = 0, p0 = 0, q0 = 0;
    int64_t pix0 = 0;
    if constexpr (KH == 3) {
      if (live) {
        const uint32_t P = (uint32_t)(pbeg + st);
        img = (int)fdiv(P, g.dppi);
        const uint32_t rem = P - (uint32_t)img * (uint32_t)g.ppi;
        const uint32_t pri = fdiv(rem, g.dpcols);
        p0 = (int)pri * PR;
        q0 = (int)(rem - pri * (uint32_t)g.pcols) * PC;
      }
      pix0 = ((int64_t)img * a.h + p0) * a.w + q0;
    } else {
      pix0 = live ? (int64_t)(pbeg + st) * Sh::NP : 0;
    }
    const __amdgpu_buffer_rsrc_t rd = hrsrc(a.dy + pix0 * a.dy_pix);
    // the halo's origin (p0 - 1, q0 - 1); the step's first pixel in the 1x1 form
    const __amdgpu_buffer_rsrc_t rx = hrsrc(a.x + (KH == 3 ? pix0 - a.w - 1 : pix0) * a.x_pix);
#pragma unroll
    for (int u = 0; u < LW; ++u) {
      const int n = wave + 8 * u;
      bool inside;
      if constexpr (KH == 3) {
        const int pr1 = (int)(lpos[u] & 0xffffu), pc1 = (int)(lpos[u] >> 16);
        inside = live && (unsigned)(p0 + pr1 - 1) < (unsigned)a.h && (unsigned)(q0 + pc1 - 1) < (unsigned)a.w;
      } else {
        inside = live && pix0 + (int64_t)lpos[u] < a.m;
      }
      const uint32_t vo = inside ? loff[u] : kOobH;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(n < NDY ? rd : rx, (hlds_void_t*)(Sg + n * 1024), 16, vo, 0, 0, 0);
    }
  };

  // Transposing reads: in each 16-lane group lane j reads 4 channels of pixel j / 4 of a
  // 4-pixel row group and lane i receives channel i of those 4 pixels; two reads (pixels
  // +0..3, +4..7) make a fragment of 8 pixels, lanes 32..63 the next 8.
  const int g16 = (lane >> 4) & 1, j16 = lane & 15;
  const int lm = 8 * (lane >> 5) + (j16 >> 2);  // this lane's pixel within a 16-pixel slice (first read)
  uint32_t aoff[OB];  // dy: byte offset of this lane's 4 channels of block ob in pixel row lm
#pragma unroll
  for (int ob = 0; ob < OB; ++ob) {
    if constexpr (RB == 192) {
      aoff[ob] = (uint32_t)(lm * 192 + ob * 64 + 32 * g16 + 8 * (j16 & 3));
    } else {
      const int slot = (ob * 4 + 2 * g16 + ((j16 & 3) >> 1)) ^ (4 * ((lm >> 1) & 1));
      aoff[ob] = (uint32_t)(lm * 128 + slot * 16 + 8 * (j16 & 1));
    }
  }
  // halo: the pixel this lane reads at slice ks, read rd is patch pixel m = 16 ks + 4 rd +
  // lm, at halo position m + 2 (m / PC) for tap (0, 0).  For PC = 16, 8 and 4 the patch row
  // m / PC splits into a compile-time part (16 ks + 4 rd) / PC and a lane part (0, the
  // lane's half, or twice it), so the position is a lane constant plus a compile-time
  // offset.
  const int lrow = PC == 16 ? 0 : (PC == 8 ? (lane >> 5) : 2 * (lane >> 5));
  const uint32_t lhalo = (uint32_t)((lm + (KH - 1) * lrow) * HRB);
  auto hoff = [&](uint32_t lb, int ks, int rd) __attribute__((always_inline)) -> uint32_t {
    const int b = 16 * ks + 4 * rd;
    return lb + (uint32_t)((b + (KH - 1) * (b / PC)) * HRB);
  };
  // this wave's run of blocks t = wq R .. wq R + R - 1 (block t: output block t % OB,
  // column block t / OB); the column blocks it touches start at cb_lo
  const int cb_lo = (wq * R) / OB;
  const int phase = (wq * R) % OB;
  uint32_t boff[NCB];  // halo: tap shift + channel offset of this lane's 16-column group per touched column block
#pragma unroll
  for (int i = 0; i < NCB; ++i) {
    int col = (cb_lo + i) * 32 + 16 * g16;
    if (col > Sh::NCOL - 16) col = Sh::NCOL - 16;  // past the last column: any valid pixel (the block is not stored)
    const int tap = col / CK, cc = col - tap * CK;
    boff[i] = (uint32_t)(((tap / KH) * HW + tap % KH) * HRB + (cc + 4 * (j16 & 3)) * 2);
  }

  // The accumulators live in the accumulation registers: an operand naming that register
  // class tells the compiler this kernel uses them, so it selects the MFMA form that keeps
  // its results there and the 16-register tuples do not crowd the vector registers.
  asm volatile("" ::"a"(0));
  f32x16 acc[R];
#pragma unroll
  for (int i = 0; i < R; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;

  auto rd2 = [&](const unsigned char* p0, const unsigned char* p1) __attribute__((always_inline)) -> u32x4 {
    const hv4s_t r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((hlds_v4s_t*)p0);
    const hv4s_t r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((hlds_v4s_t*)p1);
    const hv2u_t lo = __builtin_bit_cast(hv2u_t, r0), hi = __builtin_bit_cast(hv2u_t, r1);
    u32x4 f;
    f[0] = lo.x;
    f[1] = lo.y;
    f[2] = hi.x;
    f[3] = hi.y;
    return f;
  };
  // this half's slices of the staged patch, ks = PAR, PAR + 2, ...: the fragments of the
  // next slice are read while the current one multiplies (two fragment buffers; a
  // scheduling barrier per slice keeps the compiler from hoisting more reads, whose
  // registers it does not have)
  // `after_first` runs once the first slice's fragment reads are issued (the next stage's
  // load issue then overlaps their latency)
  auto compute = [&](auto sc, auto phc, auto parc, auto&& after_first) __attribute__((always_inline)) {
    constexpr int PH = decltype(phc)::value, PAR = decltype(parc)::value;
    constexpr int NK = (KS - PAR + 1) / 2;
    const unsigned char* Sg = stage(sc);
    const unsigned char* Hs = Sg + NDY * 1024;
    // the lane parts of the addresses, opaque to the compiler here: otherwise it hoists
    // every (slice, read, block) address out of the step loop
    uint32_t la[OB], lb[NCB];
#pragma unroll
    for (int ob = 0; ob < OB; ++ob) {
      la[ob] = aoff[ob];
      asm volatile("" : "+v"(la[ob]));
    }
#pragma unroll
    for (int i = 0; i < NCB; ++i) {
      lb[i] = lhalo + boff[i];
      asm volatile("" : "+v"(lb[i]));
    }
    u32x4 af0[OB], bf0[NCB], af1[OB], bf1[NCB];
    auto load = [&](int ks, u32x4* af, u32x4* bf) __attribute__((always_inline)) {
#pragma unroll
      for (int ob = 0; ob < OB; ++ob) {
        const unsigned char* p = Sg + la[ob] + 16 * ks * RB;
        af[ob] = rd2(p, p + 4 * RB);
      }
#pragma unroll
      for (int i = 0; i < NCB; ++i) bf[i] = rd2(Hs + hoff(lb[i], ks, 0), Hs + hoff(lb[i], ks, 1));
    };
    auto mma = [&](const u32x4* af, const u32x4* bf) __attribute__((always_inline)) {
#pragma unroll
      for (int jj = 0; jj < R; ++jj) acc[jj] = mfma32x32x16(af[(PH + jj) % OB], bf[(PH + jj) / OB], acc[jj]);
    };
    load(PAR, af0, bf0);
    __builtin_amdgcn_sched_barrier(0);
    after_first();
    static_for<0, NK>([&](auto ic) {
      constexpr int i = decltype(ic)::value;
      if constexpr ((i & 1) == 0) {
        if constexpr (i + 1 < NK) load(PAR + 2 * (i + 1), af1, bf1);
        mma(af0, bf0);
      } else {
        if constexpr (i + 1 < NK) load(PAR + 2 * (i + 1), af0, bf0);
        mma(af1, bf1);
      }
      __builtin_amdgcn_sched_barrier(0);
    });
  };
  auto sync = [&]() __attribute__((always_inline)) {
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(Sh::PENDING) : "memory");
  };
  // The main loop for one (phase, half) pair; step kt reads stage kt mod S and refills the
  // stage read last step with step kt + S - 1.  Half h takes slices ks = h, h + 2, ...
  // (for an odd slice count half 0 takes one more; each SIMD runs one wave of each half,
  // so its MFMA work per step is the same either way).
  auto main_loop = [&](auto phc, auto parc) __attribute__((always_inline)) {
    auto step = [&](auto uc, int kt) __attribute__((always_inline)) {
      constexpr int u = decltype(uc)::value;
      sync();
      compute(uc, phc, parc, [&]() __attribute__((always_inline)) { issue(IcH<(u + S - 1) % S>{}, kt + S - 1); });
    };
    static_for<0, S - 1>([&](auto ic) { issue(ic, decltype(ic)::value); });
    int kb = 0;
    for (; kb + S <= nsteps; kb += S) static_for<0, S>([&](auto ic) { step(ic, kb + decltype(ic)::value); });
    static_for<0, S - 1>([&](auto ic) {
      if (kb + decltype(ic)::value < nsteps) step(ic, kb + decltype(ic)::value);
    });
  };
  if (phase == 0) {
    if (half == 0) main_loop(IcH<0>{}, IcH<0>{});
    else main_loop(IcH<0>{}, IcH<1>{});
  } else if (OB > 1 && phase == 1) {
    if (half == 0) main_loop(IcH<1>{}, IcH<0>{});
    else main_loop(IcH<1>{}, IcH<1>{});
  } else if constexpr (OB > 2) {
    if (half == 0) main_loop(IcH<2>{}, IcH<0>{});
    else main_loop(IcH<2>{}, IcH<1>{});
  }
  // loads issued past the last step must land before the stages are reused
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  // The halves' exchange through the stages: half 1 hands over blocks jj < J0, half 0
  // blocks jj >= J0; entry (wave run wq, block jj) holds 16 fp32 x 64 lanes as four
  // 1 KiB rows of float4.
  constexpr int J0 = (R + 1) / 2;
  auto entry = [&](int jj) __attribute__((always_inline)) -> uint32_t {
    const int e = wq * R + jj;
    const int k = e / Sh::EPS;
    uint32_t b = lds_u32(sS0);
    static_for<1, S>([&](auto ic) {
      if (k == decltype(ic)::value) b = lds_u32(stage(ic));
    });
    return b + (uint32_t)((e - k * Sh::EPS) * 4096 + lane * 16);
  };
#pragma unroll
  for (int jj = 0; jj < R; ++jj) {
    if ((half == 1) != (jj < J0)) continue;
    const uint32_t ad = entry(jj);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      f32x4 v;
      v[0] = acc[jj][4 * q];
      v[1] = acc[jj][4 * q + 1];
      v[2] = acc[jj][4 * q + 2];
      v[3] = acc[jj][4 * q + 3];
      *(hlds_f4_t*)(uintptr_t)(ad + q * 1024) = v;
    }
  }
  __syncthreads();
  float* out = a.out + (a.splits > 1 ? (int64_t)bz * a.co * a.ktot : 0);
  const bool acc_in = a.splits == 1 && a.accumulate;
#pragma unroll
  for (int jj = 0; jj < R; ++jj) {
    if ((half == 0) != (jj < J0)) continue;
    const uint32_t ad = entry(jj);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 v = *(hlds_f4_t*)(uintptr_t)(ad + q * 1024);
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[jj][4 * q + e] += v[e];
    }
    const int t = wq * R + jj;
    if (t >= T) continue;
    const int ob = t % OB, cb = t / OB;
    const int col = cb * 32 + (lane & 31);
    const int tap = col / CK, cc = col - tap * CK;
    if (tap >= KH * KH || c0 + cc >= a.ci) continue;
    const int k = tap * a.ci + c0 + cc;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int o = o0 + ob * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      if (o >= a.co) continue;
      float* p = out + (int64_t)o * a.ktot + k;
      const float val = acc[jj][r];
      *p = acc_in ? *p + val : val;
    }
  }
  (void)CB;
}

struct WhCfg {
  int ob, ck, pr, pc, kh;
};

// the output-channel tile that pads c_out least, 96 rows on a tie
int wh_ob(int co) {
  const int pad2 = (co + 63) / 64 * 64 - co, pad3 = (co + 95) / 96 * 96 - co;
  return pad3 <= pad2 ? 3 : 2;
}

// The configuration for a problem, or ob = 0 where the kernel does not apply.
WhCfg wgrad_halo_cfg(const WgradArgs& a) {
  WhCfg c{0, 0, 0, 0, 0};
  if (a.ho != a.h || a.wo != a.w || a.sh != 1 || a.sw != 1) return c;
  if (a.co % 8 != 0 || a.x_pix % 8 != 0 || a.dy_pix % 8 != 0 || a.ci < 32) return c;
#ifdef NUMBAT_TUNING
  if (const char* e = getenv("NUMBAT_WH_OFF")) {
    if (atoi(e)) return c;
  }
#endif
  if (a.kh == 1 && a.kw == 1 && a.ph == 0 && a.pw == 0) {
    // 1x1: steps of 64 consecutive pixels; the largest chunk of 288, 192, 144 or 96 input
    // channels that divides c_in
    int ck = 0;
    for (const int k : {288, 192, 144, 96})
      if (ck == 0 && a.ci % k == 0) ck = k;
    if (ck == 0 || a.m >= (1ll << 36)) return c;
#ifdef NUMBAT_TUNING
    if (const char* e = getenv("NUMBAT_WH1_OFF")) {
      if (atoi(e)) return c;
    }
    if (const char* e = getenv("NUMBAT_WH1_MAXCI")) {
      if (a.ci > atoi(e)) return c;
    }
#endif
    c.ob = wh_ob(a.co);
    c.ck = ck;
    c.pr = 1;
    c.pc = 64;
    c.kh = 1;
    return c;
  }
  if (a.kh != 3 || a.kw != 3 || a.ph != 1 || a.pw != 1) return c;
  int ck = 0;
  if (a.ci % 32 == 0) ck = 32;
  else if (a.ci % 48 == 0) ck = 48;
  else return c;
  int pr = 0, pc = 0;
  if (a.h % 8 == 0 && a.w % 16 == 0) pr = 8, pc = 16;
  else if (a.h % 20 == 0 && a.w % 8 == 0) pr = 20, pc = 8;
  else if (a.h % 20 == 0 && a.w % 4 == 0) pr = 20, pc = 4;
  else return c;
  // offsets within one image (plus its halo) are 32-bit
  const int64_t pix = a.x_pix > a.dy_pix ? a.x_pix : a.dy_pix;
  if (((int64_t)a.h * a.w + 2 * (int64_t)a.w + 2) * pix * 2 >= (1ll << 31) - (1ll << 24)) return c;
  c.ob = ck == 32 ? wh_ob(a.co) : 2;
  c.ck = ck;
  c.pr = pr;
  c.pc = pc;
  c.kh = 3;
  return c;
}

int64_t wh_npatch(const WgradArgs& a, const WhCfg& c) {
  return c.kh == 1 ? (a.m + 63) / 64 : (int64_t)a.n * (a.h / c.pr) * (a.w / c.pc);
}

template <int OB, int CK, int PR, int PC, int S, int KH>
hipError_t launch_wh(const WgradArgs& a, const WhGeom& g, dim3 grid, hipStream_t s) {
  NUMBAT_LAUNCH((wgrad_halo_kernel<OB, CK, PR, PC, S, KH>), grid, dim3(512), 0, s, a, g);
  return hipGetLastError();
}

// stages: as many as the LDS holds with one block per CU (at least enough to hold the
// halves' exchange)
template <int OB, int CK>
hipError_t launch_wh_patch(const WgradArgs& a, const WhCfg& c, const WhGeom& g, dim3 grid, hipStream_t s) {
#ifdef NUMBAT_TUNING
  if (c.pr == 8 && c.pc == 16 && getenv("NUMBAT_WH_S3")) return launch_wh<OB, CK, 8, 16, 3, 3>(a, g, grid, s);
#endif
  if (c.pr == 8 && c.pc == 16) return launch_wh<OB, CK, 8, 16, 4, 3>(a, g, grid, s);
  if (c.pr == 20 && c.pc == 8) return launch_wh<OB, CK, 20, 8, 3, 3>(a, g, grid, s);
  if (c.pr == 20 && c.pc == 4) return launch_wh<OB, CK, 20, 4, (OB == 3 && CK == 32) ? 5 : 6, 3>(a, g, grid, s);
  return hipErrorInvalidValue;
}

template <int OB>
hipError_t launch_wh_1x1(const WgradArgs& a, const WhCfg& c, const WhGeom& g, dim3 grid, hipStream_t s) {
  switch (c.ck) {
    case 288: return launch_wh<OB, 288, 1, 64, 3, 1>(a, g, grid, s);
    case 192: return launch_wh<OB, 192, 1, 64, 4, 1>(a, g, grid, s);
    case 144: return launch_wh<OB, 144, 1, 64, 5, 1>(a, g, grid, s);
    case 96: return launch_wh<OB, 96, 1, 64, 6, 1>(a, g, grid, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

bool wgrad_halo_plan(const WgradArgs& a, int* splits, int64_t* patches_per_split) {
  const WhCfg c = wgrad_halo_cfg(a);
  if (c.ob == 0) return false;
  const int64_t npatch = wh_npatch(a, c);
  if (npatch >= (1ll << 30)) return false;
  const int64_t tiles = (int64_t)((a.co + 32 * c.ob - 1) / (32 * c.ob)) * ((a.ci + c.ck - 1) / c.ck);
  // Blocks: about 160.  One block fills a CU (all of its LDS and registers), and the
  // weight gradients run beside the backward's main chain on a second stream: grids that
  // leave that chain CUs made the two-stream step faster though the kernel alone is slower
  // (configuration 4 at batch 16: 256 blocks 8.91 ms per step, 192 8.73, 160 8.54, 128
  // 8.57, against 8.75 with the general kernel on every layer, same host); fewer blocks
  // also write fewer partials.
  int64_t slots = 160;
#ifdef NUMBAT_TUNING
  if (const char* e = getenv("NUMBAT_WH_SLOTS")) slots = atoi(e);
#endif
  int64_t sp = tiles < slots ? slots / tiles : 1;
  if (sp > npatch) sp = npatch;
  // partials at most 64 MiB
  const int64_t part_bytes = (int64_t)a.co * c.kh * c.kh * a.ci * 4;
  while (sp > 1 && sp * part_bytes > (64ll << 20)) --sp;
  const int64_t pps = (npatch + sp - 1) / sp;
  *patches_per_split = pps;
  *splits = (int)((npatch + pps - 1) / pps);
  return true;
}

hipError_t wgrad_halo_launch(const WgradArgs& args, hipStream_t s) {
  WgradArgs a = args;
  const WhCfg c = wgrad_halo_cfg(a);
  if (c.ob == 0 || a.ktot != c.kh * c.kh * a.ci || a.rows_per_split < 1) return hipErrorInvalidValue;
  a.remap = 1;
  WhGeom g;
  g.pcols = c.kh == 3 ? a.w / c.pc : 1;
  g.ppi = c.kh == 3 ? (a.h / c.pr) * g.pcols : 1;
  g.npatch = (int32_t)wh_npatch(a, c);
  g.pps = (int32_t)a.rows_per_split;
  g.dppi = make_fastdiv((uint32_t)g.ppi);
  g.dpcols = make_fastdiv((uint32_t)g.pcols);
  if ((int64_t)a.splits * g.pps < g.npatch) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((a.co + 32 * c.ob - 1) / (32 * c.ob)), (unsigned)((a.ci + c.ck - 1) / c.ck),
                  (unsigned)a.splits);
  trace_begin(KC_WGRAD);
  hipError_t e;
  if (c.kh == 1) e = c.ob == 3 ? launch_wh_1x1<3>(a, c, g, grid, s) : launch_wh_1x1<2>(a, c, g, grid, s);
  else if (c.ck == 48) e = launch_wh_patch<2, 48>(a, c, g, grid, s);
  else if (c.ob == 3) e = launch_wh_patch<3, 32>(a, c, g, grid, s);
  else e = launch_wh_patch<2, 32>(a, c, g, grid, s);
  trace_end(KC_WGRAD);
  return e;
}

}  // namespace numbat
