"""The Python binding rejects tensors whose dtype or shape differs from what the C ABI
would read or write (it receives bare pointers and could not tell), before anything
is launched: each call below raises, and the output tensor it was given keeps its
sentinel contents."""
import pytest
import torch

import paper_2609_39329_amd as pkv

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def t(shape, dt=torch.float32, fill=0.5):
    return torch.full(shape, fill, dtype=dt, device=DEV)


def bf(shape):
    return t(shape, torch.bfloat16)


def untouched(x, fill):
    torch.cuda.synchronize()
    return bool((x == fill).all().item())


M, Hq, Hkv, dh, N, B, d = 8, 4, 2, 64, 40, 12, 256


def test_attention_wrappers_reject_mismatches():
    Q, K, V = bf((M, Hq, dh)), bf((Hkv, N, dh)), bf((Hkv, N, dh))
    O = t((M, Hq * dh), fill=7.0)
    idx = torch.arange(B, dtype=torch.int32, device=DEV)
    cases = [
        (TypeError, lambda: pkv.attend_full(Q, K.float(), V, O=O)),            # K dtype != Q
        (ValueError, lambda: pkv.attend_full(Q, K, V[:, :N - 1], O=O)),         # V shape != K
        (ValueError, lambda: pkv.attend_full(Q, K, V, O=t((M, Hq * dh + 1), fill=7.0))),
        (TypeError, lambda: pkv.attend_full(Q, K, V, O=O.double())),
        (TypeError, lambda: pkv.attend_compressed(Q, K, V, idx=idx.long(), O=O)),
        (ValueError, lambda: pkv.attend_compressed(Q, K, V, idx=idx.view(3, 4), O=O)),  # 3 != Hkv
        (ValueError, lambda: pkv.attend_compressed(Q, K, V, idx=idx.view(2, 6),
                                                   counts=torch.ones(3, dtype=torch.int32,
                                                                     device=DEV), O=O)),
        (ValueError, lambda: pkv.attend_chunk(Q, K, V, bf((Hkv, M + 1, dh)), bf((Hkv, M, dh)), O=O)),
        (TypeError, lambda: pkv.attend_cache(Q, K, V, bias=t((Hkv, N)).double(), O=O)),
        (ValueError, lambda: pkv.attend_cache(Q, K, V, bias=t((Hkv, N + 1)), O=O)),
        (ValueError, lambda: pkv.attend_cache(Q, K.to(torch.int8), V.to(torch.int8),
                                              kv_format=pkv.KV_MXINT8, O=O)),   # exponents missing
    ]
    for exc, call in cases:
        with pytest.raises(exc):
            call()
    assert untouched(O, 7.0)


def test_statistics_and_solve_wrappers_reject_mismatches():
    X, T = t((M, d)), t((M, d))
    G, C = t((d, d), fill=3.0), t((d, d), fill=3.0)
    W = bf((d, d))
    Tout = t((M, d), fill=3.0)
    cases = [
        (TypeError, lambda: pkv.compute_targets(X, X.double(), W, T=Tout)),
        (ValueError, lambda: pkv.compute_targets(X, X, bf((d + 1, d)), T=Tout)),
        (ValueError, lambda: pkv.compute_targets(X, X, W, T=t((M, d - 4), fill=3.0))),
        # a float32 G with F64 accumulation would be written as doubles out of bounds
        (TypeError, lambda: pkv.accumulate_normal_eq(X, T, G=G, C=C, acc=pkv.F64)),
        (ValueError, lambda: pkv.accumulate_normal_eq(X, T, G=t((d, d + 1), fill=3.0), C=C)),
        (ValueError, lambda: pkv.accumulate_normal_eq(X, t((M + 1, d)), G=G, C=C)),
        (TypeError, lambda: pkv.solve_patch(G, C.double(), 0.1)),               # C dtype != G
        (ValueError, lambda: pkv.solve_patch(t((d, d + 1)), C, 0.1)),
        (ValueError, lambda: pkv.solve_patch(G, C, 0.1, dW=t((d, d - 1), fill=3.0))),
        (TypeError, lambda: pkv.solve_patch(G, C, 0.1, info=torch.zeros(1, device=DEV))),
        (ValueError, lambda: pkv.low_rank_patch(t((d + 2, d + 2)), C, r=8)),
        (ValueError, lambda: pkv.mlp_features(X, bf((d, 512)), bf((d, 508)))),
        (TypeError, lambda: pkv.propagate_student(t((M, 512)), bf((512, d)), t((512, d)).double(), X)),
        (ValueError, lambda: pkv.compute_block_targets(t((M, 512)), t((M, 512)), bf((512, d)),
                                                       X, t((M, d + 1)))),
    ]
    for exc, call in cases:
        with pytest.raises(exc):
            call()
    assert untouched(G, 3.0) and untouched(C, 3.0) and untouched(Tout, 3.0)


def test_layer_patch_wrapper_rejects_mismatches():
    Hq2, dh2 = 4, 64
    dd = Hq2 * dh2
    Q, K, V = bf((M, Hq2, dh2)), bf((Hkv, N, dh2)), bf((Hkv, N, dh2))
    idx = torch.arange(B, dtype=torch.int32, device=DEV)
    dW = t((dd, dd), fill=9.0)
    cases = [
        (ValueError, lambda: pkv.compute_layer_patch(Q, K, V, bf((dd, dd + 1)), idx=idx, dW=dW)),
        (TypeError, lambda: pkv.compute_layer_patch(Q, K, V, t((dd, dd)), idx=idx, dW=dW)),
        (ValueError, lambda: pkv.compute_layer_patch(Q, K, V, bf((dd, dd)), Kc=bf((Hkv, B, dh2)),
                                                     Vc=bf((Hkv, B + 1, dh2)), dW=dW)),
        (ValueError, lambda: pkv.compute_layer_patch(Q, K, V, bf((dd, dd)), dW=dW)),  # no cache
        (TypeError, lambda: pkv.compute_layer_patch(Q, K, V, bf((dd, dd)), idx=idx,
                                                    dW=dW.double())),
    ]
    for exc, call in cases:
        with pytest.raises(exc):
            call()
    assert untouched(dW, 9.0)
