"""The C ABI from several threads at once (calls are stateless, and
cat_last_error is per thread): host-side transform builds and weight
quantizations run concurrently give the sequential results bit for bit,
and each thread reads its own last error after another thread has failed
differently.  Runs on the CPU."""
import threading

import numpy as np

import paper_2603_04359_amd as cat
from oracle import cat_oracle as o
from paper_2603_04359_amd import binding as B


def _job(seed):
    rng = np.random.default_rng(seed)
    k, d_in, d_out = 32, 256, 96
    X = (rng.standard_normal((2048, d_in)) * np.exp(rng.standard_normal(d_in))).astype(np.float32)
    W = (rng.standard_normal((d_out, d_in)) / np.sqrt(d_in)).astype(np.float32)
    S = o.second_moment(X)
    blocks = np.stack([S[b * k:(b + 1) * k, b * k:(b + 1) * k] for b in range(d_in // k)])

    def run():
        T, Te, Wp = cat.cat_build_transform(blocks, W, k, B.CAT_BUILD_CAT, B.CAT_BF16,
                                            want_exact=True, n_threads=2)
        codes, s_w = cat.cat_quantize_weights(Wp, 4)
        return T, Te, Wp, codes, s_w
    return run


def test_concurrent_host_calls_match_sequential():
    jobs = [_job(s) for s in range(6)]
    seq = [j() for j in jobs]
    out = [None] * len(jobs)
    errs = []

    def worker(i):
        try:
            for _ in range(3):
                r = jobs[i]()
                assert all(np.array_equal(a, b) for a, b in zip(r, seq[i]))
            out[i] = True
        except Exception as e:            # reported below, on the main thread
            errs.append((i, e))

    ts = [threading.Thread(target=worker, args=(i,)) for i in range(len(jobs))]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert not errs, errs
    assert all(out)


def test_last_error_is_per_thread():
    L = B.lib()
    W = np.ones((4, 8), np.float64)
    codes = np.empty((4, 4), np.uint8)
    s_w = np.empty(4, np.float32)
    bar = threading.Barrier(2)
    seen = {}

    def fail(name, d_in, bits):
        rc = L.cat_quantize_weights(W.ctypes.data, 4, d_in, bits, codes.ctypes.data,
                                    s_w.ctypes.data)
        mine = L.cat_last_error().decode()
        bar.wait()                         # both threads have failed now
        bar.wait()
        seen[name] = (rc, mine, L.cat_last_error().decode())

    a = threading.Thread(target=fail, args=("bits", 8, 5))      # unsupported width
    b = threading.Thread(target=fail, args=("shape", 7, 4))     # odd d_in
    a.start(); b.start(); a.join(); b.join()
    rc_a, first_a, again_a = seen["bits"]
    rc_b, first_b, again_b = seen["shape"]
    assert rc_a == B.CAT_ERR_UNSUPPORTED and rc_b == B.CAT_ERR_INVALID_ARG
    assert "bits" in first_a and "even" in first_b
    assert again_a == first_a and again_b == first_b
