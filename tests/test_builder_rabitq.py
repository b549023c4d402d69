"""The product builder's RaBitQ codes (chimera_builder_rabitq, host code)
against the oracle's, bit for bit: the most significant bits, the packed
4-bit codes and both float32 factors of every token."""
import numpy as np
import pytest

import oracle
import synth
from paper_2608_23553_amd import ChimeraError, Builder, chimera
from util_build import product_builder
from util_corpus import corpus


@pytest.mark.parametrize("name,ndocs", [("tiny", None), ("2m-long", 300)])
def test_builder_rabitq_codes_equal_the_oracle(name, ndocs):
    w, c, k, cl = corpus(name, ndocs)
    signs = synth.rotation_signs(17)
    b = product_builder(c, w.nbits, rabitq_signs=signs)
    got = b.rabitq_sections()
    codes, g4, g1 = oracle.rabitq_encode(k, signs, 4)
    assert np.array_equal(got["bits1"], oracle.rabitq_pack1(codes, 4))
    packed4 = (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)
    assert np.array_equal(got["codes4"], packed4)
    assert np.array_equal(got["g1"].view(np.uint32), g1.view(np.uint32))
    assert np.array_equal(got["g4"].view(np.uint32), g4.view(np.uint32))
    with pytest.raises(ChimeraError) as e:
        b.save("/nonexistent/never-written")
    assert e.value.code == chimera.E_UNSUPPORTED
    b.close()


def test_builder_rabitq_arguments():
    w, c, k, cl = corpus("tiny")
    b = Builder(synth.k_to_bf16_bits(c.centroids_k), w.nbits)
    bad = synth.rotation_signs(1).copy()
    bad[5] = 0
    with pytest.raises(ChimeraError):
        b.rabitq(bad)
    b.close()
    b = product_builder(c, w.nbits)  # documents added: too late
    with pytest.raises(ChimeraError):
        b.rabitq(synth.rotation_signs(1))
    with pytest.raises(ChimeraError):
        b.rabitq_sections()
    b.close()
