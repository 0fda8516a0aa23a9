// Host-side number theory for the 2M + Ozaki-II library: the 2M moduli
// (Section 2 criterion, Section 4 greedy set) and their hybrid 3M extension
// (Section 3.2), roots of -1, the scaling
// budget and the CRT weights folded with the 2M post step (eq. 2m-post),
// stored as balanced base-2^40 limbs for the exact fp64 CRT of the CRT kernel.
#include <math.h>
#include <mutex>
#include <stdint.h>
#include <string.h>
#include <vector>

#include "o2m_internal.h"

namespace o2m {
namespace {

// ---- minimal unsigned big integer: little-endian 32-bit words -------------
struct Big {
    std::vector<uint32_t> w;
    void trim() { while (!w.empty() && w.back() == 0) w.pop_back(); }
    bool zero() const { return w.empty(); }
};

Big big_from(uint64_t v) {
    Big b;
    while (v) { b.w.push_back((uint32_t)v); v >>= 32; }
    return b;
}

Big big_mul_small(const Big &a, uint32_t s) {
    Big r;
    uint64_t carry = 0;
    for (uint32_t x : a.w) {
        uint64_t t = (uint64_t)x * s + carry;
        r.w.push_back((uint32_t)t);
        carry = t >> 32;
    }
    if (carry) r.w.push_back((uint32_t)carry);
    r.trim();
    return r;
}

// a / s, remainder in *rem
Big big_div_small(const Big &a, uint32_t s, uint32_t *rem) {
    Big q;
    q.w.assign(a.w.size(), 0);
    uint64_t r = 0;
    for (size_t i = a.w.size(); i-- > 0;) {
        uint64_t cur = (r << 32) | a.w[i];
        q.w[i] = (uint32_t)(cur / s);
        r = cur % s;
    }
    q.trim();
    if (rem) *rem = (uint32_t)r;
    return q;
}

int big_cmp(const Big &a, const Big &b) {
    if (a.w.size() != b.w.size()) return a.w.size() < b.w.size() ? -1 : 1;
    for (size_t i = a.w.size(); i-- > 0;)
        if (a.w[i] != b.w[i]) return a.w[i] < b.w[i] ? -1 : 1;
    return 0;
}

Big big_sub(const Big &a, const Big &b) {  // a >= b
    Big r;
    int64_t borrow = 0;
    for (size_t i = 0; i < a.w.size(); ++i) {
        int64_t t = (int64_t)a.w[i] - (i < b.w.size() ? b.w[i] : 0) - borrow;
        borrow = t < 0;
        r.w.push_back((uint32_t)(t + (borrow ? (1LL << 32) : 0)));
    }
    r.trim();
    return r;
}

Big big_shr(const Big &a, int bits) {
    Big r;
    int ws = bits / 32, bs = bits % 32;
    for (size_t i = ws; i < a.w.size(); ++i) {
        uint64_t lo = a.w[i];
        uint64_t hi = i + 1 < a.w.size() ? a.w[i + 1] : 0;
        r.w.push_back((uint32_t)(((hi << 32) | lo) >> bs));
    }
    r.trim();
    return r;
}

Big big_shl(const Big &a, int bits) {
    Big r;
    if (a.zero()) return r;
    const int ws = bits / 32, bs = bits % 32;
    r.w.assign(ws, 0);
    uint32_t carry = 0;
    for (uint32_t x : a.w) {
        r.w.push_back(bs ? (x << bs) | carry : x);
        carry = bs ? x >> (32 - bs) : 0;
    }
    if (carry) r.w.push_back(carry);
    r.trim();
    return r;
}

Big big_add(const Big &a, const Big &b) {
    Big r;
    uint64_t carry = 0;
    const size_t n = a.w.size() > b.w.size() ? a.w.size() : b.w.size();
    for (size_t i = 0; i < n; ++i) {
        const uint64_t t = (uint64_t)(i < a.w.size() ? a.w[i] : 0) + (i < b.w.size() ? b.w[i] : 0) + carry;
        r.w.push_back((uint32_t)t);
        carry = t >> 32;
    }
    if (carry) r.w.push_back((uint32_t)carry);
    r.trim();
    return r;
}

int big_bitlen(const Big &a) {
    if (a.zero()) return 0;
    return 32 * ((int)a.w.size() - 1) + (32 - __builtin_clz(a.w.back()));
}

double big_log2(const Big &a) {
    int bl = big_bitlen(a);
    if (bl <= 64) {
        uint64_t v = 0;
        for (size_t i = 0; i < a.w.size(); ++i) v |= (uint64_t)a.w[i] << (32 * i);
        return log2((double)v);
    }
    Big top = big_shr(a, bl - 60);
    uint64_t v = 0;
    for (size_t i = 0; i < top.w.size(); ++i) v |= (uint64_t)top.w[i] << (32 * i);
    return log2((double)v) + (bl - 60);
}

Big big_add_small(const Big &a, uint32_t s) {
    Big r = a;
    uint64_t carry = s;
    for (size_t i = 0; i < r.w.size() && carry; ++i) {
        uint64_t t = (uint64_t)r.w[i] + carry;
        r.w[i] = (uint32_t)t;
        carry = t >> 32;
    }
    if (carry) r.w.push_back((uint32_t)carry);
    return r;
}

uint64_t big_low_bits(const Big &a, int bits) {  // bits <= 64
    uint64_t v = 0;
    for (size_t i = 0; i < a.w.size() && i < 2; ++i) v |= (uint64_t)a.w[i] << (32 * i);
    return bits >= 64 ? v : (v & ((1ull << bits) - 1));
}

// Signed big integer mag * factor split into T balanced base-2^40 digits:
// d_t in [-2^39, 2^39) for t < T-1, the top digit takes the rest.
void balanced_limbs(const Big &mag, int64_t factor, int T, double *out) {
    bool neg = factor < 0;
    Big v = big_mul_small(mag, (uint32_t)(neg ? -factor : factor));
    for (int t = 0; t < T - 1; ++t) {
        int64_t d = (int64_t)big_low_bits(v, 40);
        v = big_shr(v, 40);
        if (d >= (1LL << 39)) { d -= 1LL << 40; v = big_add_small(v, 1); }
        out[t] = (double)(neg ? -d : d);
    }
    int64_t top = (int64_t)big_low_bits(v, 64);
    out[T - 1] = (double)(neg ? -top : top);
}

bool all_primes_1_mod_4(int m) {
    for (int p = 2; p * p <= m; ++p) {
        if (m % p == 0) {
            if (p % 4 != 1) return false;
            while (m % p == 0) m /= p;
        }
    }
    return m == 1 || m % 4 == 1;
}

int gcd(int a, int b) { while (b) { int t = a % b; a = b; b = t; } return a; }

int mod_inverse(int a, int m) {  // a, m coprime, m > 1
    int t = 0, nt = 1, r = m, nr = ((a % m) + m) % m;
    while (nr) {
        int q = r / nr, tmp;
        tmp = t - q * nt; t = nt; nt = tmp;
        tmp = r - q * nr; r = nr; nr = tmp;
    }
    return ((t % m) + m) % m;
}

int symmetric(int64_t x, int m) {
    int64_t r = ((x % m) + m) % m;
    return (int)(r > (m - 1) / 2 ? r - m : r);
}

std::mutex g_mu;
ModuliTable *g_tables[kMaxModuli + 1] = {};

}  // namespace

int root_of_minus_one(int m) {
    for (int s = 1; s < m; ++s)
        if (((int64_t)s * s + 1) % m == 0) return s;
    return 0;
}

int moduli_2m(int *out, int cap) {
    // Section 2: odd m whose prime factors are all 1 mod 4; Section 4: greedy
    // from 256 down, keeping m coprime to every modulus kept so far.
    int n = 0;
    int kept[64];
    for (int m = 256; m >= 3; --m) {
        if (m % 2 == 0 || !all_primes_1_mod_4(m)) continue;
        bool ok = true;
        for (int i = 0; i < n; ++i)
            if (gcd(m, kept[i]) != 1) { ok = false; break; }
        if (!ok) continue;
        kept[n++] = m;
    }
    for (int i = 0; i < n && i < cap; ++i) out[i] = kept[i];
    return n;
}

int moduli_extension(int *out, int cap) {
    // Section 3.2 (hybrid 2M / 3M): continue the greedy scan over all
    // integers, coprime to the 2M set and to every extension modulus kept.
    int kept[128];
    int n = moduli_2m(kept, 64);
    const int n2 = n;
    for (int m = 256; m >= 2; --m) {
        bool ok = true;
        for (int i = 0; i < n; ++i)
            if (gcd(m, kept[i]) != 1) { ok = false; break; }
        if (ok && n < 128) kept[n++] = m;
    }
    for (int i = n2; i < n && i - n2 < cap; ++i) out[i - n2] = kept[i];
    return n - n2;
}

const ModuliTable *moduli_table(int n) {
    if (n < 1 || n > kMaxModuli) return nullptr;
    std::lock_guard<std::mutex> lock(g_mu);
    if (g_tables[n]) return g_tables[n];

    int all[128];
    const int n2all = moduli_2m(all, 64);
    moduli_extension(all + n2all, 64);
    const int n2 = n < n2all ? n : n2all;
    ModuliTable *t = new ModuliTable();
    memset(t, 0, sizeof *t);
    t->n = n;

    Big M = big_from(1);
    for (int l = 0; l < n; ++l) M = big_mul_small(M, (uint32_t)all[l]);
    t->log2M = big_log2(M);
    t->mwords_len = (int)M.w.size();
    for (size_t i = 0; i < M.w.size() && i < 8; ++i) t->mwords[i] = M.w[i];

    // residue constants
    ResidueParams &rp = t->res;
    rp.n = n;
    rp.n2 = n2;
    for (int l = 0; l < n; ++l) {
        int m = all[l];
        rp.mod[l] = m;
        rp.root[l] = l < n2 ? root_of_minus_one(m) : 0;
        rp.inv[l] = 1.0 / (double)m;
        int64_t p26 = 1;
        for (int b = 0; b < 26; ++b) p26 = p26 * 2 % m;
        int64_t pw = 1;
        for (int d = 1; d < kMaxDigits; ++d) {          // 2^(26 d) mod m
            pw = pw * p26 % m;
            rp.cpow[l][d - 1] = (double)symmetric(pw, m);
        }
    }

    // CRT weights folded with 2^-1 (Re) and s 2^-1 (Im), eq. 2m-post; plain
    // weights for the 3M moduli of a hybrid set
    CrtParams &cp = t->crt;
    cp.n = n;
    cp.n2 = n2;
    cp.limbs = (int)ceil((t->log2M + 1.0) / kLimbBits);
    if (cp.limbs < 2) cp.limbs = 2;
    for (int l = 0; l < n; ++l) {
        int m = all[l];
        uint32_t rem;
        Big Ml = big_div_small(M, (uint32_t)m, &rem);     // M / m_l
        uint32_t Ml_mod;
        big_div_small(Ml, (uint32_t)m, &Ml_mod);
        int inv_Ml = mod_inverse((int)Ml_mod, m);
        if (l >= n2) {
            balanced_limbs(Ml, symmetric(inv_Ml, m), cp.limbs, cp.wre[l]);
            continue;
        }
        int half = (m + 1) / 2;                             // 2^-1 mod m (Section 2)
        int s = rp.root[l];
        int gre = symmetric((int64_t)inv_Ml * half, m);
        int gim = symmetric((int64_t)inv_Ml * half % m * s, m);
        balanced_limbs(Ml, gre, cp.limbs, cp.wre[l]);
        balanced_limbs(Ml, gim, cp.limbs, cp.wim[l]);
    }
    balanced_limbs(M, 1, cp.limbs, cp.mlimb);
    {
        // fl(1/M) from the top 64 bits of M
        int bl = big_bitlen(M);
        Big top = bl > 64 ? big_shr(M, bl - 64) : M;
        uint64_t v = 0;
        for (size_t i = 0; i < top.w.size(); ++i) v |= (uint64_t)top.w[i] << (32 * i);
        long double lv = (long double)v;
        if (bl > 64) lv = ldexpl(lv, bl - 64);
        cp.inv_m = (double)(1.0L / lv);
    }
    if (t->log2M < 63.5) {
        uint64_t mv = 0;
        for (size_t i = 0; i < M.w.size(); ++i) mv |= (uint64_t)M.w[i] << (32 * i);
        cp.m_lo = mv;
        cp.m_hi = 0;
        cp.h_lo = (mv - 1) / 2;
    }
    g_tables[n] = t;
    return t;
}

namespace {
// (M-1)/2 - floor(M/2^32): the largest |Re c|, |Im c| the CRT kernel recovers.
Big recoverable(const ModuliTable *t) {
    Big M;
    M.w.assign(t->mwords, t->mwords + t->mwords_len);
    M.trim();
    uint32_t r;
    Big h = big_div_small(big_sub(M, big_from(1)), 2, &r);  // (M-1)/2
    Big margin = big_shr(M, 32);
    return big_cmp(h, margin) > 0 ? big_sub(h, margin) : Big();
}
}  // namespace

bool budget_cs(const ModuliTable *t, int k, bool symmetric, int *qA, int *qB) {
    const Big hp = recoverable(t);
    uint64_t R = 0;                                 // ceil(sqrt(k/2)): 2 R^2 >= k
    while (2 * R * R < (uint64_t)(k > 0 ? k : 0)) ++R;
    for (int S = big_bitlen(hp) - 1; S >= 0; --S) {
        const int a = S / 2, b = symmetric ? a : S - a;
        // (2^a + R)(2^b + R) = 2^(a+b) + R 2^a + R 2^b + R^2
        Big v = big_shl(big_from(1), a + b);
        v = big_add(v, big_shl(big_from(R), a));
        v = big_add(v, big_shl(big_from(R), b));
        v = big_add(v, big_from(R * R));
        if (big_cmp(v, hp) <= 0) {
            *qA = a;
            *qB = b;
            return true;
        }
    }
    return false;
}

int budget(const ModuliTable *t, int k) {
    uint32_t r;
    Big bmax = recoverable(t);
    uint64_t two_k = 2ull * (uint64_t)(k > 0 ? k : 1);
    if (big_cmp(bmax, big_from(two_k)) >= 0) {
        Big q = big_div_small(bmax, (uint32_t)two_k, &r);
        return big_bitlen(q) - 1;
    }
    uint64_t b = 0;
    for (size_t i = 0; i < bmax.w.size(); ++i) b |= (uint64_t)bmax.w[i] << (32 * i);
    if (b == 0) return -1000;
    int s = 1;
    while ((b << s) < two_k) ++s;
    return -s;
}

}  // namespace o2m
