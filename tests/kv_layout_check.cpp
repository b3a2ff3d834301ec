// Host check of the KV cache block layout: both maps are bijections onto the block, and the
// fragment the attention loads for (tile, step, lane) holds the keys and dims it multiplies.
#include <cstdio>
#include <vector>
#include "kernels.h"
using namespace dvi;
int main() {
    for (int kc : {16, 32})
        for (int hd : {64, 128}) {
            const int epl = kc / 4, n = 64 * hd, ds = hd / kc, ks = 64 / kc;
            std::vector<int> seen_k(n, 0), seen_v(n, 0);
            for (int kk = 0; kk < 64; ++kk)
                for (int d = 0; d < hd; ++d) {
                    const size_t ok = kv_key_offset(kc, hd, kk, d), ov = kv_val_offset(kc, hd, kk, d);
                    if (ok >= (size_t)n || ov >= (size_t)n) { printf("out of block\n"); return 1; }
                    seen_k[ok]++;
                    seen_v[ov]++;
                }
            for (int i = 0; i < n; ++i)
                if (seen_k[i] != 1 || seen_v[i] != 1) { printf("not a bijection kc=%d hd=%d\n", kc, hd); return 1; }
            for (int l = 0; l < 64; ++l)
                for (int e = 0; e < epl; ++e) {
                    for (int t = 0; t < 4; ++t)
                        for (int st = 0; st < ds; ++st)
                            if (kv_key_offset(kc, hd, 16 * t + l % 16, st * kc + epl * (l / 16) + e) !=
                                ((size_t)(t * ds + st) * 64 + l) * epl + e) { printf("key fragment\n"); return 1; }
                    for (int dt = 0; dt < hd / 16; ++dt)
                        for (int s = 0; s < ks; ++s)
                            if (kv_val_offset(kc, hd, s * kc + epl * (l / 16) + e, 16 * dt + l % 16) !=
                                ((size_t)(dt * ks + s) * 64 + l) * epl + e) { printf("value fragment\n"); return 1; }
                }
        }
    printf("ok\n");
    return 0;
}
