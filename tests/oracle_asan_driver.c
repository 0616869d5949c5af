/*
 * Test driver for the C oracles under AddressSanitizer and
 * UndefinedBehaviorSanitizer (CPU only; built by
 * tests/test_oracle_sanitizers.py with the oracle sources linked in).
 *
 * Reads one request from argv[1], runs it through the oracle entry point it
 * names and writes the raw results to argv[2].  Every input array is read
 * into an allocation of exactly its size, so any read past the end of a job
 * table or a grid table is reported by the sanitizer.
 *
 * Request layout (native endianness, no padding):
 *   int32 kind            0 oracle_cells, 1 oracle_cells_tab, 2 proxy_oracle_cells
 *   int32 rule            partition rule (kind 0) / operators per job (kind 2)
 *   int32 n_jobs, n_layers, n_types, n_counts, n_m, n_sel, K, cuts_stride
 *   float64 tie_eps, f_ref
 *   int32 off[n_jobs+1]; float32 t, p, a, x, a2a [n_layers]; int32 batch[n_jobs]
 *   float32 speed, mem, bw_intra, bw_inter [n_types]; int32 gpn[n_types]; float32 hbm[n_types]
 *   int32 counts[n_counts]; float32 kappa[n_types*n_counts]; int32 m[n_m]; int64 ids[n_sel]
 *   float64 vol[n_types*2*K], lat[n_types*2*K]          (kind 1 only)
 * Result: kinds 0/1: float64 res[2 n_sel], int32 plan[4 n_sel],
 *   int32 cuts[n_sel cuts_stride], int32 nplans[n_sel];
 *   kind 2: float64 out[4 n_sel], int32 plan[52 n_sel].
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_cells(int n_sel, const int64_t* cells, int n_types, int n_counts, const int32_t* off,
                 const float* t, const float* p, const float* a, const float* x, const float* a2a,
                 const int32_t* batch, const float* speed, const float* mem, const float* bwi,
                 const float* bwe, const int32_t* gpn, const int32_t* counts, const float* kappa_grid,
                 const int32_t* m_values, int n_m, double tie_eps, double* res, int32_t* plan,
                 int32_t* cuts, int cuts_stride, int32_t* nplans, int rule);
int oracle_cells_tab(int n_sel, const int64_t* cells, int n_types, int n_counts, const int32_t* off,
                     const float* t, const float* p, const float* a, const float* x, const float* a2a,
                     const int32_t* batch, const float* speed, const float* mem, const float* bwi,
                     const float* bwe, const int32_t* gpn, const int32_t* counts, const float* kappa_grid,
                     const int32_t* m_values, int n_m, double tie_eps, int K, const double* vol,
                     const double* lat, double* res, int32_t* plan, int32_t* cuts, int cuts_stride,
                     int32_t* nplans);
int proxy_oracle_cells(int n_sel, const int64_t* cells, int n_types, int n_counts, const int32_t* off,
                       const float* t, const float* p, const float* a, const float* x, const float* a2a,
                       const int32_t* batch, const float* speed, const float* mem, const float* bwi,
                       const float* bwe, const int32_t* gpn, const float* hbm, const int32_t* counts,
                       const float* kappa, const int32_t* m_values, int n_m, double tie_eps, double f_ref,
                       int n_ops, double* out, int32_t* plan);

static FILE* in_file;

static void* take(size_t elem, size_t n)
{
    void* p = malloc(elem * n ? elem * n : 1);
    if (!p) {
        fprintf(stderr, "driver: out of memory\n");
        exit(3);
    }
    if (n && fread(p, elem, n, in_file) != n) {
        fprintf(stderr, "driver: short request\n");
        exit(3);
    }
    return p;
}

int main(int argc, char** argv)
{
    if (argc != 3) return 2;
    in_file = fopen(argv[1], "rb");
    if (!in_file) return 2;
    int32_t* hdr = (int32_t*)take(4, 10);
    const int kind = hdr[0], rule = hdr[1], nj = hdr[2], nl = hdr[3], nt = hdr[4], nc = hdr[5];
    const int nm = hdr[6], ns = hdr[7], K = hdr[8], stride = hdr[9];
    double* sc = (double*)take(8, 2);
    int32_t* off = (int32_t*)take(4, (size_t)nj + 1);
    float* t = (float*)take(4, (size_t)nl);
    float* p = (float*)take(4, (size_t)nl);
    float* a = (float*)take(4, (size_t)nl);
    float* x = (float*)take(4, (size_t)nl);
    float* q = (float*)take(4, (size_t)nl);
    int32_t* batch = (int32_t*)take(4, (size_t)nj);
    float* speed = (float*)take(4, (size_t)nt);
    float* mem = (float*)take(4, (size_t)nt);
    float* bwi = (float*)take(4, (size_t)nt);
    float* bwe = (float*)take(4, (size_t)nt);
    int32_t* gpn = (int32_t*)take(4, (size_t)nt);
    float* hbm = (float*)take(4, (size_t)nt);
    int32_t* counts = (int32_t*)take(4, (size_t)nc);
    float* kappa = (float*)take(4, (size_t)nt * nc);
    int32_t* ms = (int32_t*)take(4, (size_t)nm);
    int64_t* ids = (int64_t*)take(8, (size_t)ns);
    double* vol = kind == 1 ? (double*)take(8, (size_t)nt * 2 * K) : NULL;
    double* lat = kind == 1 ? (double*)take(8, (size_t)nt * 2 * K) : NULL;
    fclose(in_file);

    FILE* out = fopen(argv[2], "wb");
    if (!out) return 2;
    int rc;
    if (kind == 0 || kind == 1) {
        double* res = (double*)malloc(sizeof(double) * 2 * (size_t)ns + 8);
        int32_t* plan = (int32_t*)malloc(sizeof(int32_t) * 4 * (size_t)ns + 4);
        int32_t* cuts = (int32_t*)malloc(sizeof(int32_t) * (size_t)ns * stride + 4);
        int32_t* np = (int32_t*)malloc(sizeof(int32_t) * (size_t)ns + 4);
        if (!res || !plan || !cuts || !np) return 3;
        if (kind == 0)
            rc = oracle_cells(ns, ids, nt, nc, off, t, p, a, x, q, batch, speed, mem, bwi, bwe, gpn, counts,
                              kappa, ms, nm, sc[0], res, plan, cuts, stride, np, rule);
        else
            rc = oracle_cells_tab(ns, ids, nt, nc, off, t, p, a, x, q, batch, speed, mem, bwi, bwe, gpn, counts,
                                  kappa, ms, nm, sc[0], K, vol, lat, res, plan, cuts, stride, np);
        fwrite(res, sizeof(double), 2 * (size_t)ns, out);
        fwrite(plan, sizeof(int32_t), 4 * (size_t)ns, out);
        fwrite(cuts, sizeof(int32_t), (size_t)ns * stride, out);
        fwrite(np, sizeof(int32_t), (size_t)ns, out);
        free(res); free(plan); free(cuts); free(np);
    } else {
        double* o4 = (double*)malloc(sizeof(double) * 4 * (size_t)ns + 8);
        int32_t* plan = (int32_t*)malloc(sizeof(int32_t) * 52 * (size_t)ns + 4);
        if (!o4 || !plan) return 3;
        rc = proxy_oracle_cells(ns, ids, nt, nc, off, t, p, a, x, q, batch, speed, mem, bwi, bwe, gpn, hbm,
                                counts, kappa, ms, nm, sc[0], sc[1], rule, o4, plan);
        fwrite(o4, sizeof(double), 4 * (size_t)ns, out);
        fwrite(plan, sizeof(int32_t), 52 * (size_t)ns, out);
        free(o4); free(plan);
    }
    fclose(out);
    free(hdr); free(sc); free(off); free(t); free(p); free(a); free(x); free(q); free(batch);
    free(speed); free(mem); free(bwi); free(bwe); free(gpn); free(hbm); free(counts); free(kappa);
    free(ms); free(ids); free(vol); free(lat);
    return rc == 0 ? 0 : 4;
}
