// Subspace Adam update of SubZero+ (Eqs. 6-10, tail of Alg. 3), and the plain
// subspace SGD update it is compared with (S = Zbar, no moments; SubZero's own
// update when q = 1).
//
// One descriptor per matrix (Item) lives in the caller's workspace: small
// k_fill_items launches copy FILL_ITEMS host descriptors each into that table
// (kernel arguments only, nothing else touches host memory).  Then three
// launches cover every matrix of the call at once, so the big update kernel
// has one tail per call instead of one per group of matrices:
//   k_adam_rr   256 entries of one matrix per workgroup: Zbar = (1/q) sum_j g_j Z_j,
//               the two r x r moments (Eqs. 7-8) and the bias-corrected direction S
//               (Eq. 9, Adam form), all in float64.  S and the new moments go to
//               the workspace with one non-finite flag per workgroup; Zbar goes
//               to zbar_out.
//   k_us        Reads the item's flags: if any entry was non-finite the item is
//               skipped (state untouched).  Otherwise commits the new moments and
//               forms L = lr U S (m x rp; tiles of 128 rows, register-blocked fp32
//               FMA) and, for 16-bit W, the hi/lo split of V (n x rp); padding
//               columns are zero.  16-bit W: L and V as hi + lo bf16 pairs (x = hi +
//               lo to about 16 significant bits, with fp32's range); fp32 W: L in
//               fp32, V read as is.
//   k_update_*  W <- W - L V^T in place.
//
// bf16 or fp16 W (k_update_bf16, the W type a template parameter: it changes
// only the conversion of W to fp32 and the rounding of the result back, both
// to nearest even): memory bound -- 4 bytes of HBM traffic per weight
// against 2 r MACs.  At r = 64 that is 32 FLOP/B, above the fp32 VALU ridge
// of the chip, so the rank-r product runs on v_mfma_f32_16x16x32_bf16 as
// hi*hi + lo*hi + hi*lo (3 MFMAs per 32-deep K step).  Each wave owns a strip
// of 64 columns whose V fragments stay in registers and walks its rows 16 at a
// time; the L rows are staged once per workgroup in LDS.
//
// Every W, L and V access of k_update_bf16 is a buffer instruction whose
// descriptor covers exactly the workgroup's rows: rows past the edge and
// columns past n (given an out-of-range offset) read as zero and drop their
// stores in hardware, so the loop has no branches around memory operations
// and the compiler can count the loads in flight exactly.  W is read NS steps
// ahead and the next L chunk one chunk ahead.
#include <vector>

#include "zo_internal.h"

namespace {

constexpr int FILL_ITEMS = 16;           // descriptors per k_fill_items launch
constexpr long long MAX_PASS_WG = 1 << 22; // workgroups per launch (x 256 threads < 2^32)
constexpr int UPD_ROWS = 512;  // rows per workgroup
constexpr int UPD_COLS = 256;  // columns per workgroup (4 waves x 64)
constexpr int UPD_GROUP = 4;   // row chunks per raster group
constexpr int US_ROWS = 128;   // rows of L per k_us workgroup
constexpr unsigned OOB = 0x80000000u;  // buffer offset beyond every descriptor used here
constexpr int RSRC_CFG = 0x00020000;   // buffer descriptor word 3: 32-bit raw access

// One matrix of the call.  Pointers marked (ws) are carved from the workspace.
struct Item {
  const float* Z;
  float* M1;        // moments: read by k_adam_rr, committed by k_us
  float* M2;
  float* zbar_out;
  double* S;        // (ws) r x r
  float* M1n;       // (ws) r x r
  float* M2n;       // (ws) r x r
  int* flags;       // (ws) one per k_adam_rr workgroup of the item
  int* skip;        // (ws) set by k_us: the item had a non-finite entry
  const float* U;
  const float* V;
  void* L;          // (ws) 16-bit W: m rows of [hi (rp) | lo (rp)] bf16; fp32 W: m x rp fp32
  void* Vs;         // (ws) 16-bit W: hi then lo (2 x n x rp) bf16; unused for fp32 W
  void* W;
  float* wout;
  int m, n;
  int us_begin;     // first k_us workgroup of the item (over the whole call)
  int l_tiles;      // k_us workgroups forming L (US_ROWS rows each); then V tiles (64 rows each)
  int us_wg;        // all k_us workgroups of the item
  int up_begin;     // first update workgroup of the item
  int strips, rchunks;  // 16-bit W: 256-column strips x 512-row chunks
};

struct FillArgs {
  Item it[FILL_ITEMS];
  Item* dst;
  int* us_begin;
  int* up_begin;
  int c0, cn;
};

// Copies one group of host descriptors (kernel arguments) into the workspace
// table, one 32-bit word per thread, and fills the two workgroup-start arrays
// searched by find_item.
__global__ __launch_bounds__(256) void k_fill_items(FillArgs a) {
  constexpr int WORDS = (int)(sizeof(Item) / 4);
  static_assert(sizeof(Item) % 4 == 0, "Item must be a whole number of words");
  const uint32_t* src = (const uint32_t*)a.it;
  uint32_t* dst = (uint32_t*)(a.dst + a.c0);
  for (int x = threadIdx.x; x < a.cn * WORDS; x += 256) dst[x] = src[x];
  if (threadIdx.x < a.cn) {
    a.us_begin[a.c0 + threadIdx.x] = a.it[threadIdx.x].us_begin;
    a.up_begin[a.c0 + threadIdx.x] = a.it[threadIdx.x].up_begin;
  }
}

// The item that workgroup b belongs to: the last k with begin[k] <= b
// (begin is non-decreasing and begin[0] = 0 <= b).  A 64-way search: each
// round one load per lane and a ballot, so 240 items take two rounds.
__device__ __forceinline__ int find_item(const int* __restrict__ begin, int count, int b) {
  const int lane = threadIdx.x & 63;
  int lo = 0, len = count;
  while (len > 64) {
    const int step = (len + 63) >> 6;
    const int off = lane * step;
    const bool le = off < len && begin[lo + off] <= b;
    const int c = __popcll(__ballot(le));
    lo += (c - 1) * step;
    len = min(step, len - (c - 1) * step);
  }
  const bool le = lane < len && begin[lo + lane] <= b;
  return __builtin_amdgcn_readfirstlane(lo + __popcll(__ballot(le)) - 1);
}

struct RRArgs {
  const Item* it;
  const float* g;
  int* nonfinite_flag;
  int r, q, aw;  // aw: workgroups per item
  int sgd;       // 1: S = Zbar, no moments
  double beta1, beta2, eps_adam, bc1, bc2;
};

__global__ __launch_bounds__(256) void k_adam_rr(RRArgs a) {
  const Item it = a.it[blockIdx.x / a.aw];
  const int w = blockIdx.x % a.aw;
  const int rr = a.r * a.r;
  const int e = w * 256 + threadIdx.x;
  int bad = 0;
  if (e < rr) {
    double zb = 0.0;
    for (int j = 0; j < a.q; ++j) zb += (double)a.g[j] * (double)it.Z[(size_t)j * rr + e];
    zb /= (double)a.q;
    double s = zb;
    if (!a.sgd) {
      const double m1 = a.beta1 * (double)it.M1[e] + (1.0 - a.beta1) * zb;
      const double m2 = a.beta2 * (double)it.M2[e] + (1.0 - a.beta2) * zb * zb;
      s = (m1 / a.bc1) / (sqrt(m2 / a.bc2) + a.eps_adam);
      it.M1n[e] = (float)m1;
      it.M2n[e] = (float)m2;
    }
    if (!isfinite(zb) || !isfinite(s)) bad = 1;
    if (it.zbar_out) it.zbar_out[e] = (float)zb;
    it.S[e] = s;
  }
  bad = __syncthreads_or(bad);
  if (threadIdx.x == 0) {
    it.flags[w] = bad;
    if (bad && a.nonfinite_flag) *a.nonfinite_flag = 1;
  }
}

struct USArgs {
  const Item* it;
  const int* begin;  // us_begin of every item
  int count, r, rp, bf16, aw, sgd;
  int wg0;           // first workgroup of this launch over the whole call
  float lr;
};

// L = lr U S for rows i0 .. i0+127 of one item: 32 columns of K at a time, U
// (transposed) and S staged in LDS as fp32; each thread owns 4 rows x rp/8
// adjacent columns.  Or the hi/lo split of 64 rows of V.
template <int RPK>
__global__ __launch_bounds__(256) void k_us(USArgs a) {
  constexpr int RP = 32 * RPK;
  constexpr int CPT = RP / 8;  // columns per thread
  __shared__ __attribute__((aligned(16))) float Ut[32][US_ROWS + 4];
  __shared__ __attribute__((aligned(16))) float Sl[32][RP];
  const int b = a.wg0 + (int)blockIdx.x;
  const Item it = a.it[find_item(a.begin, a.count, b)];
  const int local = b - it.us_begin;
  const int r = a.r, tid = threadIdx.x;
  int bad = 0;
  for (int w = tid; w < a.aw; w += 256) bad |= it.flags[w];
  bad = __syncthreads_or(bad);
  if (local == 0 && tid == 0) *it.skip = bad;
  if (bad) return;
  const int rr = r * r;
  if (!a.sgd) {
    for (int e = local * 256 + tid; e < rr; e += it.us_wg * 256) {
      it.M1[e] = it.M1n[e];
      it.M2[e] = it.M2n[e];
    }
  }
  if (local < it.l_tiles) {
    const int i0 = local * US_ROWS;
    const int tr = tid >> 3, tc = tid & 7;
    float acc[4][CPT];
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
      for (int y = 0; y < CPT; ++y) acc[x][y] = 0.f;
    for (int kc = 0; kc < RPK; ++kc) {
      if (kc) __syncthreads();
      for (int x = tid; x < 32 * US_ROWS; x += 256) {
        const int i = x >> 5, kk = x & 31, t = kc * 32 + kk;
        Ut[kk][i] = (i0 + i < it.m && t < r) ? it.U[(size_t)(i0 + i) * r + t] : 0.f;
      }
      for (int x = tid; x < 32 * RP; x += 256) {
        const int kk = x / RP, c = x % RP, t = kc * 32 + kk;
        Sl[kk][c] = (t < r && c < r) ? (float)it.S[t * r + c] : 0.f;
      }
      __syncthreads();
#pragma unroll 4
      for (int kk = 0; kk < 32; ++kk) {
        const f32x4 u = *(const f32x4*)&Ut[kk][tr * 4];
        float s[CPT];
#pragma unroll
        for (int y = 0; y < CPT; y += 4) {
          const f32x4 sv = *(const f32x4*)&Sl[kk][tc * CPT + y];
          s[y] = sv[0];
          s[y + 1] = sv[1];
          s[y + 2] = sv[2];
          s[y + 3] = sv[3];
        }
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
          for (int y = 0; y < CPT; ++y) acc[x][y] = fmaf(u[x], s[y], acc[x][y]);
      }
    }
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const int i = i0 + tr * 4 + x;
      if (i >= it.m) break;
      if (a.bf16) {
        bf16_t* Lh = (bf16_t*)it.L + (size_t)i * 2 * RP + tc * CPT;
        bf16_t* Ll = Lh + RP;
#pragma unroll
        for (int y = 0; y < CPT; y += 4) {
          float v[4], lo[4];
#pragma unroll
          for (int z = 0; z < 4; ++z) {
            v[z] = a.lr * acc[x][y + z];
            lo[z] = v[z] - bf16_to_f32(f32_to_bf16(v[z]));
          }
          *(u32x2*)(Lh + y) = (u32x2){pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
          *(u32x2*)(Ll + y) = (u32x2){pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3])};
        }
      } else {
        // fp32 W keeps L unpadded: m x rp with rp == r.
        float* Lf = (float*)it.L + (size_t)i * a.rp;
#pragma unroll
        for (int y = 0; y < CPT; ++y)
          if (tc * CPT + y < a.rp) Lf[tc * CPT + y] = a.lr * acc[x][y];
      }
    }
  } else {
    constexpr int G = RP / 8;  // 8-column groups per row
    const int k0 = (local - it.l_tiles) * 64;
    bf16_t* Vh = (bf16_t*)it.Vs;
    bf16_t* Vl = Vh + (size_t)it.n * RP;
    for (int x = tid; x < 64 * G; x += 256) {
      const int row = k0 + x / G, c0 = (x % G) * 8;
      if (row >= it.n) break;
      float v[8], lo[8];
      const float* vr = it.V + (size_t)row * r + c0;
      if (r % 4 == 0 && c0 + 8 <= r && (uintptr_t)it.V % 16 == 0) {  // two 16-byte loads
        const f32x4 a0 = *(const f32x4*)vr, a1 = *(const f32x4*)(vr + 4);
        v[0] = a0[0]; v[1] = a0[1]; v[2] = a0[2]; v[3] = a0[3];
        v[4] = a1[0]; v[5] = a1[1]; v[6] = a1[2]; v[7] = a1[3];
      } else {
#pragma unroll
        for (int z = 0; z < 8; ++z) v[z] = c0 + z < r ? vr[z] : 0.f;
      }
#pragma unroll
      for (int z = 0; z < 8; ++z) lo[z] = v[z] - bf16_to_f32(f32_to_bf16(v[z]));
      *(u32x4*)(Vh + (size_t)row * RP + c0) = (u32x4){pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                                      pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
      *(u32x4*)(Vl + (size_t)row * RP + c0) =
          (u32x4){pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]), pack_bf16x2(lo[4], lo[5]),
                  pack_bf16x2(lo[6], lo[7])};
    }
  }
}

struct UpdArgs {
  const Item* it;
  const int* begin;  // up_begin of every item
  int count, r, rp;
  int wg0;           // first workgroup of this launch over the whole call
  int pass_wg;       // workgroups of this launch
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, (int)bytes, RSRC_CFG);
}
__device__ __forceinline__ u32x4 bload(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
}
__device__ __forceinline__ void bstore(__amdgpu_buffer_rsrc_t r, unsigned off, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)off, 0, 0);
}

__device__ __forceinline__ u32x2 bload2(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0);
}
__device__ __forceinline__ void bstore2(__amdgpu_buffer_rsrc_t r, unsigned off, u32x2 v) {
  __builtin_amdgcn_raw_buffer_store_b64(v, r, (int)off, 0, 0);
}

// Workgroup tile: UPD_ROWS rows x 256 columns (4 waves x 64 columns), walked in
// chunks of CH = 16 NS rows.  Per chunk: the chunk's L rows (loaded a chunk
// earlier into registers) go to LDS, the next chunk's L is requested, and each
// of the NS steps multiplies 16 rows, stores them and requests the same step of
// the next chunk.  The MFMA takes L rows as its A operand and V columns as its
// B operand, column j of tile t being W column 4 j + t of the wave's strip: a
// lane ends with 4 ADJACENT columns of rows 4 g .. 4 g + 3 (g = lane / 16),
// so each memory instruction of a wave covers 4 rows x 128 contiguous bytes --
// whole cache lines.  The prologue issues range-dropped stores in place of each
// step's stores so that the count of memory operations between a load and its
// use is the same on entry as in the steady state.
template <int RPK, bool HOOK, bool WF16>
__global__ __launch_bounds__(256) void k_update_bf16(UpdArgs a) {
  constexpr int RP = 32 * RPK;
  constexpr int NS = RPK == 1 ? 4 : 2;  // W prefetch depth in 16-row steps
  constexpr int CH = 16 * NS;           // rows per L chunk
  constexpr int LROW = RP * 4 + 16;     // bytes per staged L row [hi | lo] (+16: conflict-free reads)
  constexpr int V16 = RP * 4 / 16;      // 16-byte pieces per L row
  constexpr int NL = CH * V16 / 256;    // L pieces per thread per chunk
  static_assert(NL * 256 == CH * V16, "L chunk must split evenly over 256 threads");
  __shared__ __attribute__((aligned(16))) char Ls[CH * LROW];
  // The hardware deals workgroup w to XCD w % 8.  Each XCD gets a contiguous
  // range of tiles, rastered in groups of UPD_GROUP row chunks: within a group
  // the row chunk runs fastest, then the strip.  The ~32 workgroups an XCD runs
  // at once then cover about 4 row chunks x 8 strips, so each chunk's L rows
  // (128 KB at r = 64) and each strip's V fragments (64 KB) come from its L2
  // after the first read, instead of once per workgroup.
  const int w = blockIdx.x, nt = a.pass_wg;
  const int xcd = w & 7, widx = w >> 3;
  const int lt = a.wg0 + xcd * (nt >> 3) + min(xcd, nt & 7) + widx;
  const Item it = a.it[find_item(a.begin, a.count, lt)];
  if (*it.skip) return;
  const int local = lt - it.up_begin;
  const int per_group = UPD_GROUP * it.strips;
  const int grp = local / per_group;
  const int gsize = min(UPD_GROUP, it.rchunks - grp * UPD_GROUP);
  const int rem = local - grp * per_group;
  const int rchunk = grp * UPD_GROUP + rem % gsize;
  const int strip = rem / gsize;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const int m = it.m, n = it.n;
  const int col0 = strip * UPD_COLS + wave * 64;
  const int row0 = rchunk * UPD_ROWS;
  const int rows = min(UPD_ROWS, m - row0);
  const int nch = (rows + CH - 1) / CH;

  const __amdgpu_buffer_rsrc_t rl =
      rsrc((const bf16_t*)it.L + (size_t)row0 * 2 * RP, (unsigned)rows * RP * 4);
  const __amdgpu_buffer_rsrc_t rv = rsrc(it.Vs, (unsigned)n * RP * 4);
  bf16_t* Wt = (bf16_t*)it.W + (size_t)row0 * n;
  const __amdgpu_buffer_rsrc_t rw = rsrc(Wt, (unsigned)rows * n * 2);
  __amdgpu_buffer_rsrc_t ro = rw;
  // Items without a hook buffer get an empty descriptor: their hook stores are dropped.
  if (HOOK) ro = it.wout ? rsrc(it.wout + (size_t)row0 * n, (unsigned)rows * n * 4) : rsrc(Wt, 0u);

  // V fragments of the strip (B operand): column j = l16 of tile t is W column
  // col0 + 4 j + t.
  const int cb = col0 + 4 * l16;
  bf16x8 vh[RPK][4], vl[RPK][4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
#pragma unroll
    for (int kk = 0; kk < RPK; ++kk) {
      const bool ok = cb + t < n;
      const unsigned off = (unsigned)(((cb + t) * RP + kk * 32 + g * 8) * 2);
      vh[kk][t] = __builtin_bit_cast(bf16x8, bload(rv, ok ? off : OOB));
      vl[kk][t] = __builtin_bit_cast(bf16x8, bload(rv, ok ? off + (unsigned)n * RP * 2 : OOB));
    }
  }
  // The fragments are complete before the loop: a wait inside it would
  // otherwise count them as possibly in flight on every iteration.
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)

  // This lane's W pieces: rows 4 g + v (v = 0..3) of each step, columns cb .. cb+3
  // (n % 8 == 0, so the 4 columns are all in range or all out).
  const unsigned stepw = (unsigned)(16 * n * 2);
  unsigned wo[4], ho[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    wo[v] = cb < n ? (unsigned)(((4 * g + v) * n + cb) * 2) : OOB;
    ho[v] = cb < n ? (unsigned)(((4 * g + v) * n + cb) * 4) : OOB;
  }

  // This thread's L pieces: (row, 16-byte column) of a chunk.
  unsigned lo_g[NL];
  int lo_s[NL];
#pragma unroll
  for (int x = 0; x < NL; ++x) {
    const int p = tid + 256 * x;
    const int rrow = p / V16, c16 = p % V16;
    lo_g[x] = (unsigned)(rrow * RP * 4 + c16 * 16);
    lo_s[x] = rrow * LROW + c16 * 16;
  }
  const unsigned chunk_l = (unsigned)(CH * RP * 4);

  u32x4 lreg[NL];
  u32x2 wb[NS][4];
#pragma unroll
  for (int x = 0; x < NL; ++x) lreg[x] = bload(rl, lo_g[x]);
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    // Distinct offsets keep the compiler from merging the dropped stores.
#pragma unroll
    for (int v = 0; v < 4; ++v) bstore2(rw, OOB + 32 * s + 8 * v, (u32x2){0u, 0u});
    if (HOOK) {
#pragma unroll
      for (int v = 0; v < 4; ++v) bstore(ro, OOB + 64 * s + 16 * v, (u32x4){0u, 0u, 0u, 0u});
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) wb[s][v] = bload2(rw, wo[v] + s * stepw);
  }

  for (int c = 0; c < nch; ++c) {
    __syncthreads();  // every wave is done with the previous chunk's L
#pragma unroll
    for (int x = 0; x < NL; ++x) *(u32x4*)(Ls + lo_s[x]) = lreg[x];
    __syncthreads();
#pragma unroll
    for (int x = 0; x < NL; ++x) lreg[x] = bload(rl, lo_g[x] + (c + 1) * chunk_l);
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      bf16x8 uh[RPK], ul[RPK];
#pragma unroll
      for (int kk = 0; kk < RPK; ++kk) {
        const char* lp = Ls + (s * 16 + l16) * LROW + (kk * 32 + g * 8) * 2;
        uh[kk] = *(const bf16x8*)lp;
        ul[kk] = *(const bf16x8*)(lp + RP * 2);
      }
      f32x4 acc[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        acc[t] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < RPK; ++kk) {
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(uh[kk], vh[kk][t], acc[t], 0, 0, 0);
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ul[kk], vh[kk][t], acc[t], 0, 0, 0);
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(uh[kk], vl[kk][t], acc[t], 0, 0, 0);
        }
      }
      // acc[t][v] is row 4 g + v, column cb + t.
      const unsigned d = (unsigned)(c * NS + s) * stepw;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const uint32_t w0 = wb[s][v][0], w1 = wb[s][v][1];
        float n0, n1, n2, n3;
        if constexpr (WF16) {
          n0 = f16_to_f32((uint16_t)w0) - acc[0][v];
          n1 = f16_to_f32((uint16_t)(w0 >> 16)) - acc[1][v];
          n2 = f16_to_f32((uint16_t)w1) - acc[2][v];
          n3 = f16_to_f32((uint16_t)(w1 >> 16)) - acc[3][v];
          bstore2(rw, wo[v] + d, (u32x2){pack_f16x2(n0, n1), pack_f16x2(n2, n3)});
        } else {
          n0 = __uint_as_float(w0 << 16) - acc[0][v];
          n1 = __uint_as_float(w0 & 0xffff0000u) - acc[1][v];
          n2 = __uint_as_float(w1 << 16) - acc[2][v];
          n3 = __uint_as_float(w1 & 0xffff0000u) - acc[3][v];
          bstore2(rw, wo[v] + d, (u32x2){pack_bf16x2(n0, n1), pack_bf16x2(n2, n3)});
        }
        if (HOOK) bstore(ro, ho[v] + 2 * d, __builtin_bit_cast(u32x4, (f32x4){n0, n1, n2, n3}));
      }
      const unsigned dn = (unsigned)((c + 1) * NS + s) * stepw;
#pragma unroll
      for (int v = 0; v < 4; ++v) wb[s][v] = bload2(rw, wo[v] + dn);
    }
  }
}

// fp32 W: one thread per weight, fp32 FMA over the r columns.
__global__ __launch_bounds__(256) void k_update_f32(UpdArgs a) {
  const int b = a.wg0 + (int)blockIdx.x;
  const Item it = a.it[find_item(a.begin, a.count, b)];
  if (*it.skip) return;
  const long long e = (long long)(b - it.up_begin) * 256 + threadIdx.x;
  if (e >= (long long)it.m * it.n) return;
  const int i = (int)(e / it.n), c = (int)(e % it.n);
  const float* L = (const float*)it.L;  // m x rp (rp = r)
  const float* V = it.V;               // n x r
  float d = 0.f;
  for (int t = 0; t < a.r; ++t) d = fmaf(L[(size_t)i * a.rp + t], V[(size_t)c * a.r + t], d);
  float* W = (float*)it.W;
  const float nv = W[e] - d;
  W[e] = nv;
  if (it.wout) it.wout[e] = nv;
}

struct Layout {
  size_t s, mom, flags, skip, L, Vs, total;
};
Layout item_layout(int m, int n, int r, int rp, int bf16, int aw) {
  Layout l;
  l.s = zo_align256((size_t)r * r * 8);
  l.mom = zo_align256((size_t)r * r * 4);
  l.flags = zo_align256((size_t)aw * 4);
  l.skip = 256;
  l.L = zo_align256((size_t)m * rp * 4);  // bf16: hi+lo; fp32: one
  l.Vs = bf16 ? zo_align256((size_t)n * rp * 4) : 0;
  l.total = l.s + 2 * l.mom + l.flags + l.skip + l.L + l.Vs;
  return l;
}

template <int RPK, bool WF16>
void launch_update_w16(bool hook, int wg, hipStream_t stream, const UpdArgs& pa) {
  if (hook)
    hipLaunchKernelGGL((k_update_bf16<RPK, true, WF16>), dim3(wg), dim3(256), 0, stream, pa);
  else
    hipLaunchKernelGGL((k_update_bf16<RPK, false, WF16>), dim3(wg), dim3(256), 0, stream, pa);
}

template <int RPK>
void launch_update_bf16(bool hook, bool wf16, int wg, hipStream_t stream, const UpdArgs& pa) {
  if (wf16)
    launch_update_w16<RPK, true>(hook, wg, stream, pa);
  else
    launch_update_w16<RPK, false>(hook, wg, stream, pa);
}

}  // namespace

int zo_update_launch(int count, const zo_update_item* items, int w_dtype, int r, int q,
                     const float* g, int t, float lr, float beta1, float beta2, float eps_adam,
                     int sgd, int* nonfinite_flag, void* ws, size_t ws_bytes, hipStream_t stream,
                     size_t* ws_needed) {
  // 16-bit W (bf16 or fp16) takes the MFMA path: L and V as hi+lo bf16 pairs.
  const int bf16 = w_dtype != ZO_F32;
  const bool wf16 = w_dtype == ZO_F16;
  const int rp = bf16 ? (r + 31) / 32 * 32 : r;
  const int aw = (r * r + 255) / 256;
  // Workspace: the descriptor table and the two workgroup-start arrays, then
  // each item's regions.
  size_t need = zo_align256((size_t)count * sizeof(Item)) + 2 * zo_align256((size_t)count * 4);
  for (int i = 0; i < count; ++i) need += item_layout(items[i].m, items[i].n, r, rp, bf16, aw).total;
  if (ws_needed) *ws_needed = need;
  if (!ws) return ZO_OK;
  if (ws_bytes < need) {
    zo_set_error("update: workspace %zu bytes < required %zu", ws_bytes, need);
    return ZO_ERR_WORKSPACE;
  }
  if (bf16 && rp / 32 > 4) {
    zo_set_error("update: r = %d above %d", r, ZO_MAX_RANK);
    return ZO_ERR_UNSUPPORTED;
  }
  if (count <= 0) return ZO_OK;
  WsCarver wc(ws);
  Item* dtab = (Item*)wc.take((size_t)count * sizeof(Item));
  int* us_begin = (int*)wc.take((size_t)count * 4);
  int* up_begin = (int*)wc.take((size_t)count * 4);
  std::vector<Item> tab((size_t)count);
  long long us_total = 0, up_total = 0;
  bool hook = false;
  for (int k = 0; k < count; ++k) {
    const zo_update_item& src = items[k];
    const Layout lay = item_layout(src.m, src.n, r, rp, bf16, aw);
    Item& it = tab[k];
    it.Z = src.Z;
    it.M1 = src.M1;
    it.M2 = src.M2;
    it.zbar_out = src.zbar_out;
    it.S = (double*)wc.take(lay.s);
    it.M1n = (float*)wc.take(lay.mom);
    it.M2n = (float*)wc.take(lay.mom);
    it.flags = (int*)wc.take(lay.flags);
    it.skip = (int*)wc.take(lay.skip);
    it.L = wc.take(lay.L);
    it.Vs = lay.Vs ? wc.take(lay.Vs) : nullptr;
    it.U = src.U;
    it.V = src.V;
    it.W = src.W;
    it.wout = src.w_f32_out;
    it.m = src.m;
    it.n = src.n;
    it.l_tiles = (src.m + US_ROWS - 1) / US_ROWS;
    it.us_wg = it.l_tiles + (bf16 ? (src.n + 63) / 64 : 0);
    it.us_begin = (int)us_total;
    us_total += it.us_wg;
    it.up_begin = (int)up_total;
    if (bf16) {
      it.strips = (src.n + UPD_COLS - 1) / UPD_COLS;
      it.rchunks = (src.m + UPD_ROWS - 1) / UPD_ROWS;
      up_total += (long long)it.strips * it.rchunks;
    } else {
      it.strips = it.rchunks = 1;
      up_total += ((long long)src.m * src.n + 255) / 256;
    }
    if (us_total >= (1LL << 31) || up_total >= (1LL << 31)) {
      zo_set_error("update: too many workgroups for one call (item %d); split the items", k);
      return ZO_ERR_UNSUPPORTED;
    }
    hook = hook || src.w_f32_out;
  }
  if ((long long)count * aw > MAX_PASS_WG) {
    zo_set_error("update: %d items above the %lld per call", count, MAX_PASS_WG / aw);
    return ZO_ERR_UNSUPPORTED;
  }
  int st;
  for (int c0 = 0; c0 < count; c0 += FILL_ITEMS) {
    FillArgs fa{};
    fa.dst = dtab;
    fa.us_begin = us_begin;
    fa.up_begin = up_begin;
    fa.c0 = c0;
    fa.cn = count - c0 < FILL_ITEMS ? count - c0 : FILL_ITEMS;
    for (int k = 0; k < fa.cn; ++k) fa.it[k] = tab[c0 + k];
    hipLaunchKernelGGL(k_fill_items, dim3(1), dim3(256), 0, stream, fa);
    if ((st = zo_hip_status(hipGetLastError(), "k_fill_items")) != ZO_OK) return st;
  }

  RRArgs ra{};
  ra.it = dtab;
  ra.g = g;
  ra.nonfinite_flag = nonfinite_flag;
  ra.r = r;
  ra.q = q;
  ra.aw = aw;
  ra.sgd = sgd;
  ra.beta1 = beta1;
  ra.beta2 = beta2;
  ra.eps_adam = eps_adam;
  ra.bc1 = 1.0 - pow((double)beta1, (double)t);
  ra.bc2 = 1.0 - pow((double)beta2, (double)t);
  hipLaunchKernelGGL(k_adam_rr, dim3((unsigned)(count * aw)), dim3(256), 0, stream, ra);
  if ((st = zo_hip_status(hipGetLastError(), "k_adam_rr")) != ZO_OK) return st;

  USArgs ua{};
  ua.it = dtab;
  ua.begin = us_begin;
  ua.count = count;
  ua.r = r;
  ua.rp = rp;
  ua.bf16 = bf16;
  ua.aw = aw;
  ua.sgd = sgd;
  ua.lr = lr;
  for (long long w0 = 0; w0 < us_total; w0 += MAX_PASS_WG) {
    const long long nw = us_total - w0 < MAX_PASS_WG ? us_total - w0 : MAX_PASS_WG;
    ua.wg0 = (int)w0;
    const dim3 grid((unsigned)nw);
    switch ((rp + 31) / 32) {
      case 1: hipLaunchKernelGGL(k_us<1>, grid, dim3(256), 0, stream, ua); break;
      case 2: hipLaunchKernelGGL(k_us<2>, grid, dim3(256), 0, stream, ua); break;
      case 3: hipLaunchKernelGGL(k_us<3>, grid, dim3(256), 0, stream, ua); break;
      default: hipLaunchKernelGGL(k_us<4>, grid, dim3(256), 0, stream, ua); break;
    }
    if ((st = zo_hip_status(hipGetLastError(), "k_us")) != ZO_OK) return st;
  }

  UpdArgs pa{};
  pa.it = dtab;
  pa.begin = up_begin;
  pa.count = count;
  pa.r = r;
  pa.rp = rp;
  for (long long w0 = 0; w0 < up_total; w0 += MAX_PASS_WG) {
    const long long nw = up_total - w0 < MAX_PASS_WG ? up_total - w0 : MAX_PASS_WG;
    pa.wg0 = (int)w0;
    pa.pass_wg = (int)nw;
    if (!bf16) {
      hipLaunchKernelGGL(k_update_f32, dim3((unsigned)nw), dim3(256), 0, stream, pa);
    } else {
      switch (rp / 32) {
        case 1: launch_update_bf16<1>(hook, wf16, (int)nw, stream, pa); break;
        case 2: launch_update_bf16<2>(hook, wf16, (int)nw, stream, pa); break;
        case 3: launch_update_bf16<3>(hook, wf16, (int)nw, stream, pa); break;
        default: launch_update_bf16<4>(hook, wf16, (int)nw, stream, pa); break;
      }
    }
    if ((st = zo_hip_status(hipGetLastError(), "k_update")) != ZO_OK) return st;
  }
  return ZO_OK;
}
