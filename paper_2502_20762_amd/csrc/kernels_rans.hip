// Entropy coding of the quantised latent (Fig. 4 "AE" / "AD", Fig. 6): rANS
// (Duda 2013, range variant: 32-bit state in [2^16, 2^32), 16-bit words,
// M = 2^16) on quantised-scale Gaussian tables.
//
// A stream is 8192 symbols coded by the 64 lanes of one wave in lock step:
// symbol i of the stream belongs to lane i % 64 at step i / 64.  At every
// (step, sub-symbol) the lanes that move a word do so in lane order (ballot +
// popcount give each its slot), so a stream is one contiguous run of words.
// An escaped symbol (|q| beyond its table) continues with one 16-bit field
// of frequency 1: 32768 * sign + |q| - R - 1.
//
// Every coder kernel first stages what its sequential loop touches into LDS
// with direct global->LDS loads issued back to back and one wait (the tables,
// the stream's symbols and scale indices, the decoder also the stream's
// words), so the loop over the 128 steps never waits on global memory.
//
// k_rans_encode  one wave per stream: encodes backwards into the stream's
//                scratch slot, words ending at the slot's end
// k_rans_pack    one workgroup per stream: copies the words into the
//                container; workgroup 0 writes the header and length table
// k_rans_decode  one wave per stream: checks the container, decodes forward,
//                every word read bounded by the stream's length; flags a
//                truncated or inconsistent stream instead of reading past it
#include "common.hpp"
#include "internal.hpp"

namespace nc {

namespace {

constexpr uint32_t kRansL = 1u << 16;

// Direct global->LDS load of 4 bytes per lane: lane l's bytes land at
// lds_wave_base + 4 l.  Callers wait with s_waitcnt vmcnt before reading.
__device__ __forceinline__ void dma4(const void* g, const void* lds_wave_base) {
  const uint32_t m = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)lds_wave_base;
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off" ::"v"(g), "s"(m) : "memory", "m0");
}

// Stages n16 16-byte chunks from g into LDS at lds (one wave, 1 KiB per load
// instruction).
__device__ __forceinline__ void stage16(const void* g, void* lds, int n16, int lane) {
  for (int i = 0; i < n16; i += 64)
    if (i + lane < n16) dma16((const uint8_t*)g + 16 * (i + lane), (uint8_t*)lds + 16 * i);
}

// x / f and x mod f for 1 <= f < 2^16 and x < f 2^16 (the quotient is below
// 2^16): the fp32 estimate x * rcp(f) is within 2^-6 of x / f (relative error
// at most about 2^-22 on a quotient below 2^16), so its truncation is off by
// at most one and a single correction each way makes it exact.
__device__ __forceinline__ uint32_t divmod16(uint32_t x, uint32_t f, uint32_t& r) {
  const uint32_t q0 = (uint32_t)((float)x * __builtin_amdgcn_rcpf((float)f));
  const int32_t r0 = (int32_t)(x - __umul24(q0, f));
  const bool under = r0 < 0, over = r0 >= (int32_t)f;
  r = (uint32_t)(r0 + (under ? (int32_t)f : 0) - (over ? (int32_t)f : 0));
  return q0 + (over ? 1u : 0u) - (under ? 1u : 0u);
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += (uint32_t)__shfl_xor((int)v, off, 64);
  return v;
}

__device__ __forceinline__ uint32_t wave_or(uint32_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v |= (uint32_t)__shfl_xor((int)v, off, 64);
  return v;
}

}  // namespace

// One wave (workgroup) per stream.  The table lookup of a step (symbol and
// scale index, then R and the scale's first start, then the entry) runs three
// steps ahead of the state chain, one stage per step, so none of its LDS reads
// is waited for on the chain.
__global__ __launch_bounds__(64) void k_rans_encode(const int16_t* q, const uint8_t* kidx, int64_t n,
                                                  const uint16_t* tab, uint16_t* scratch, int64_t max_words,
                                                  uint32_t* lens) {
  __shared__ __align__(16) uint16_t st[kTabEncU16];
  __shared__ __align__(16) int16_t sq[kRansStream];
  __shared__ __align__(16) uint8_t sk[kRansStream];
  const int lane = threadIdx.x;
  const int64_t s = blockIdx.x;
  const int64_t base = s * kRansStream;
  const int cnt = (int)min((int64_t)kRansStream, n - base);
  const int steps = (cnt + 63) / 64;
  stage16(tab, st, kTabEncU16 / 8, lane);
  const int nq = cnt / 8, nk = cnt / 16;  // whole 16-byte chunks; q and k are 16-byte aligned
  stage16(q + base, sq, nq, lane);
  stage16(kidx + base, sk, nk, lane);
  if (8 * nq + lane < cnt) sq[8 * nq + lane] = q[base + 8 * nq + lane];
  if (16 * nk + lane < cnt) sk[16 * nk + lane] = kidx[base + 16 * nk + lane];
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  const uint16_t* sst = st + kTabStarts;
  // positions past cnt read values that are never used; every index stays
  // inside the tables
  int aq = 0, ak = 0;                            // stage A: symbol, scale index
  int bq = 0, bR = 0, bo = 0;                    // stage B: symbol, R, first start
  uint32_t cc = 0, cf = 1;                       // stage C: start, frequency,
  int cq = 0, cR = 0;                            //          symbol, R
  auto stage_a = [&](int u) {
    if (u >= 0) {
      aq = sq[u * 64 + lane];
      ak = sk[u * 64 + lane];
    }
  };
  auto stage_b = [&]() {
    const int k = min(ak, kCoderScales - 1);
    bq = aq;
    bR = st[4 * k];
    bo = st[4 * k + 1];
  };
  auto stage_c = [&]() {
    const int i = (bq < -bR || bq > bR) ? 2 * bR + 1 : bq + bR;
    const uint32_t c0 = sst[bo + i], c1 = sst[bo + i + 1];
    cc = c0;
    cf = (c1 - c0) & 0xFFFFu;
    cq = bq;
    cR = bR;
  };
  stage_a(steps - 1);
  stage_b();
  stage_c();
  stage_a(steps - 2);
  stage_b();
  stage_a(steps - 3);
  uint16_t* end = scratch + (s + 1) * max_words;
  const uint64_t below = (1ull << lane) - 1;
  int p = 0;  // words written, counted back from the end
  uint32_t x = kRansL;
  for (int t = steps - 1; t >= 0; --t) {
    const int li = t * 64 + lane;
    const bool act = li < cnt;
    const uint32_t c = cc, f = act ? cf : 1u;
    const int qv = cq, R = cR;
    stage_c();
    stage_b();
    stage_a(t - 3);
    const bool esc = act && (qv < -R || qv > R);
    if (__ballot(esc)) {
      // the field follows the escape in decoding order, so it is coded first;
      // with frequency 1 every escaped state moves a word out
      const uint64_t m = __ballot(esc);
      const int cw = (int)__popcll(m);  // __popcll is unsigned: keep the slot arithmetic signed
      if (esc) {
        const uint32_t fld = (qv < 0 ? 32768u : 0u) + (uint32_t)(abs(qv) - R - 1);
        end[(int)__popcll(m & below) - (p + cw)] = (uint16_t)(x & 0xFFFFu);
        x = (x & 0xFFFF0000u) | fld;
      }
      p += cw;
    }
    const bool emit = act && x >= (f << 16);
    const uint64_t m = __ballot(emit);
    const int cw = (int)__popcll(m);
    if (emit) end[(int)__popcll(m & below) - (p + cw)] = (uint16_t)(x & 0xFFFFu);
    x = emit ? x >> 16 : x;
    p += cw;
    uint32_t r;
    const uint32_t qd = divmod16(x, f, r);
    x = act ? (qd << 16) + r + c : x;
  }
  // the 64 final states open the stream: lane l at words 2l (high) and 2l + 1
  end[-(p + 128) + 2 * lane] = (uint16_t)(x >> 16);
  end[-(p + 128) + 2 * lane + 1] = (uint16_t)(x & 0xFFFFu);
  p += 128;
  if (lane == 0) lens[s] = (uint32_t)p;
}

// One workgroup per stream: the stream's place in the container is the sum of
// the lengths before it (every workgroup sums them itself, so no separate scan
// pass); workgroup 0 also writes the header and the length table.
__global__ __launch_bounds__(256) void k_rans_pack(const uint16_t* scratch, int64_t max_words, const uint32_t* lens,
                                                 int64_t n, uint8_t* out, uint64_t* nbytes) {
  __shared__ uint32_t sa[4], stot[4];
  const int ns = (int)((n + kRansStream - 1) / kRansStream);
  const int s = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t a = 0, tot = 0;
  for (int i = threadIdx.x; i < ns; i += 256) {
    const uint32_t v = lens[i];
    tot += v;
    a += i < s ? v : 0u;
  }
  a = wave_sum(a);
  tot = wave_sum(tot);
  if (lane == 0) {
    sa[wave] = a;
    stot[wave] = tot;
  }
  __syncthreads();
  a = sa[0] + sa[1] + sa[2] + sa[3];
  tot = stot[0] + stot[1] + stot[2] + stot[3];
  const uint32_t len = lens[s];
  const uint16_t* src = scratch + (int64_t)(s + 1) * max_words - len;
  uint16_t* dst = (uint16_t*)(out + rans_payload_offset(ns)) + a;
  for (uint32_t i = threadIdx.x; i < len; i += 256) dst[i] = src[i];
  if (s == 0) {
    uint16_t* ltab = (uint16_t*)(out + kRansHeader);
    for (int i = threadIdx.x; i < ns; i += 256) ltab[i] = (uint16_t)lens[i];
    if (threadIdx.x == 0) {
      uint32_t* h = (uint32_t*)out;
      h[0] = kRansMagic;
      h[1] = kRansVersion;
      h[2] = (uint32_t)n;
      h[3] = (uint32_t)kRansStream;
      h[4] = (uint32_t)ns;
      if (ns & 1) ltab[ns] = 0;  // pad to 4 bytes
      *nbytes = (uint64_t)rans_payload_offset(ns) + 2ull * tot;
    }
  }
}

// One wave (workgroup) per stream.  LDS holds the whole coder table block,
// the stream's scale indices and the stream's words (word i at sw[par + i],
// par the parity of the stream's start, so that whole dwords can be staged).
// Every workgroup checks the container header and sums the length table up to
// its stream itself.  Each writes its error bits to errs[s]; the last one to
// finish (a ticket on *count, which it resets) merges them into *status_out.
__global__ __launch_bounds__(64) void k_rans_decode(const uint8_t* in, uint64_t in_bytes, const uint8_t* kidx,
                                                  int64_t n, const uint16_t* tab, uint32_t* errs, uint32_t* count,
                                                  int16_t* q, int32_t* status_out) {
  __shared__ __align__(16) uint16_t st[kTabU16];
  __shared__ __align__(16) uint8_t sk[kRansStream];
  __shared__ __align__(16) uint16_t sw[kRansMaxWords + 2];
  const int lane = threadIdx.x;
  const int s = blockIdx.x;
  const int ns = (int)((n + kRansStream - 1) / kRansStream);
  const int64_t base = (int64_t)s * kRansStream;
  const int cnt = (int)min((int64_t)kRansStream, n - base);
  const int steps = (cnt + 63) / 64;
  stage16(tab, st, kTabU16 / 8, lane);
  const int nk = cnt / 16;  // k is 16-byte aligned
  stage16(kidx + base, sk, nk, lane);
  if (16 * nk + lane < cnt) sk[16 * nk + lane] = kidx[base + 16 * nk + lane];
  // container check (wave-uniform: every lane reads the same words; all loads
  // issued before the first use)
  bool bad = in_bytes < (uint64_t)rans_payload_offset(ns);
  const uint16_t* ltab = (const uint16_t*)(in + kRansHeader);
  uint32_t a = 0, tot = 0;
  if (!bad) {
    const uint32_t* h = (const uint32_t*)in;
    const uint32_t h0 = h[0], h1 = h[1], h2 = h[2], h3 = h[3], h4 = h[4];
#pragma unroll 4
    for (int i = lane; i < ns; i += 64) {
      const uint32_t v = ltab[i];
      tot += v;
      a += i < s ? v : 0u;
    }
    bad = (h0 != kRansMagic) | (h1 != kRansVersion) | (h2 != (uint32_t)n) | (h3 != (uint32_t)kRansStream) |
          (h4 != (uint32_t)ns);
  }
  // the sums are wave-uniform; readfirstlane puts them in scalar registers (the
  // LDS destination of the word staging below goes through M0)
  a = (uint32_t)__builtin_amdgcn_readfirstlane((int)wave_sum(a));
  tot = (uint32_t)__builtin_amdgcn_readfirstlane((int)wave_sum(tot));
  if (!bad && (uint64_t)rans_payload_offset(ns) + 2ull * tot > in_bytes) bad = true;
  uint32_t err = bad ? 1u : 0u;
  uint32_t len = bad ? 0u : (uint32_t)ltab[s];
  if (len > (uint32_t)kRansMaxWords) {
    err |= 2;
    len = 0;
  }
  if (len < 128) err |= 2;
  // the stream's words are u16 indices [g0, g1) of the container
  const uint64_t g0 = (uint64_t)(rans_payload_offset(ns) / 2) + a, g1 = g0 + len;
  const int par = (int)(g0 & 1);
  {
    // whole dwords d0 .. d1 - 1 inside [g0, g1); dword d lands at sw[2 (d - g0 / 2)]
    const uint64_t d0 = (g0 + 1) / 2, d1 = g1 / 2;
    const int nd = d1 > d0 ? (int)(d1 - d0) : 0;
    const uint32_t* src = (const uint32_t*)in + d0;
    uint16_t* dst = sw + 2 * (d0 - g0 / 2);
    for (int i = 0; i < nd; i += 64)
      if (i + lane < nd) dma4(src + i + lane, dst + 2 * i);
    const uint16_t* in16 = (const uint16_t*)in;
    if (lane == 0 && len > 0 && par) sw[1] = in16[g0];                          // odd first word
    if (lane == 1 && len > 0 && (g1 & 1)) sw[par + len - 1] = in16[g1 - 1];   // odd last word
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  const uint16_t* sst = st + kTabStarts;
  const uint16_t* sbk = st + kTabBuckets;
  const uint64_t below = (1ull << lane) - 1;
  auto word = [&](uint32_t i) -> uint32_t { return i < len ? (uint32_t)sw[par + i] : 0u; };
  uint32_t x = (word(2 * lane) << 16) | word(2 * lane + 1);
  uint32_t pos = 128;
  // lane-ordered renormalisation reads of the lanes in need
  auto refill = [&](bool need) {
    const uint64_t m = __ballot(need);
    if (need) {
      const uint32_t i = pos + (uint32_t)__popcll(m & below);
      if (i >= len) err |= 2;
      x = (x << 16) | word(i);
    }
    pos += (uint32_t)__popcll(m);
  };
  // table coordinates that do not depend on the state run ahead of the state
  // chain: the scale index two steps, its R, first start and tail counts one
  // step (positions past cnt read values that are never used; every index
  // stays inside the tables).  The index is clamped where it is used, not where
  // it is loaded, so that the load is not waited for until the next step.
  const uint2* shead = (const uint2*)st;  // scale j: (R | first << 16, T | U << 16)
  int k1 = min((int)sk[lane], kCoderScales - 1);
  int k2 = steps > 1 ? (int)sk[64 + lane] : 0;
  uint2 h1 = shead[k1];
  for (int t = 0; t < steps; ++t) {
    const int li = t * 64 + lane;
    const bool act = li < cnt;
    const int row = 257 * k1;
    const int R = (int)(h1.x & 0xFFFFu), o = (int)(h1.x >> 16);
    const uint32_t T = h1.y & 0xFFFFu, U = h1.y >> 16;
    k1 = min(k2, kCoderScales - 1);
    h1 = shead[k1];
    if (t + 2 < steps) k2 = sk[li + 128];
    const uint32_t slot = x & 0xFFFFu;
    // slots in the leading or trailing run of frequency-1 entries map to
    // their entry directly; elsewhere the bucket bounds the entry holding the
    // slot, most buckets hold at most one entry boundary, settled by the next
    // start, and the rest are searched
    const bool head = slot < T, tail = slot >= 65536u - U;
    int lo = sbk[row + (slot >> 8)];
    const int hi = sbk[row + (slot >> 8) + 1];
    const uint32_t v0 = sst[o + lo], v1 = sst[o + lo + 1], v2 = sst[o + lo + 2];
    const bool up = hi > lo && v1 <= slot;
    uint32_t c = up ? v1 : v0, cn = up ? v2 : v1;
    lo += up ? 1 : 0;
    if (!head && !tail && hi > lo && cn <= slot) {
      int h = hi;
      while (lo < h) {
        const int mid = (lo + h + 1) >> 1;
        if (sst[o + mid] <= slot) lo = mid;
        else h = mid - 1;
      }
      c = sst[o + lo];
      cn = sst[o + lo + 1];
    }
    if (head || tail) {
      lo = head ? (int)slot : 2 * R + 2 - 65536 + (int)slot;
      c = slot;
      cn = slot + 1;
    }
    const uint32_t f = (cn - c) & 0xFFFFu;
    const bool esc = act && lo == 2 * R + 1;
    if (act) x = f * (x >> 16) + slot - c;
    refill(act && x < kRansL);
    int qv = lo - R;
    if (__ballot(esc)) {
      const uint32_t fld = x & 0xFFFFu;
      if (esc) x >>= 16;
      refill(esc);
      if (esc) {
        const int mag = R + 1 + (int)(fld & 32767u);
        qv = (fld >> 15) ? -mag : mag;
      }
    }
    if (act) q[base + li] = (int16_t)max(min(qv, 32767), -32768);
  }
  if (!bad && (x != kRansL || pos != len)) err |= 4;
  err = wave_or(err);
  uint32_t ticket = 0;
  if (lane == 0) {
    errs[s] = err;
    __threadfence();
    ticket = atomicAdd(count, 1u);
  }
  ticket = (uint32_t)__shfl((int)ticket, 0, 64);
  if (ticket == (uint32_t)ns - 1) {  // every other stream has published its bits
    __threadfence();
    uint32_t all = 0;
    for (int i = lane; i < ns; i += 64) all |= __hip_atomic_load(errs + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    all = wave_or(all);
    if (lane == 0) {
      if (status_out) *status_out = (int32_t)all;
      __hip_atomic_store(count, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

hipError_t launch_rans_encode(const int16_t* q, const uint8_t* k, int64_t n, const uint16_t* tab, uint16_t* scratch,
                              int64_t max_words, uint32_t* lens, uint8_t* out, uint64_t* nbytes, hipStream_t st) {
  const int64_t ns = (n + kRansStream - 1) / kRansStream;
  if (ns <= 0 || ns > 65535) return hipErrorInvalidValue;
  launch(k_rans_encode, dim3((unsigned)ns), dim3(64), st, q, k, n, tab, scratch, max_words, lens);
  launch(k_rans_pack, dim3((unsigned)ns), dim3(256), st, (const uint16_t*)scratch, max_words, (const uint32_t*)lens, n,
         out, nbytes);
  return hipGetLastError();
}

hipError_t launch_rans_decode(const uint8_t* in, uint64_t in_bytes, const uint8_t* k, int64_t n, const uint16_t* tab,
                              uint32_t* errs, uint32_t* count, int16_t* q, int32_t* status_out, hipStream_t st) {
  const int64_t ns = (n + kRansStream - 1) / kRansStream;
  if (ns <= 0 || ns > 65535) return hipErrorInvalidValue;
  launch(k_rans_decode, dim3((unsigned)ns), dim3(64), st, in, in_bytes, k, n, tab, errs, count, q, status_out);
  return hipGetLastError();
}

}  // namespace nc
