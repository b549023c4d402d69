"""The library's offline index builder (host C++) against the oracle's own
quantiser, codes, packing and posting lists (Sec. 3.1 offline index building)."""
import os
import struct

import numpy as np
import pytest

import oracle
import synth
from paper_2608_23553_amd import Builder, ChimeraError, Index, chimera
from util_build import product_builder
from util_corpus import corpus, oracle_index


@pytest.mark.parametrize("name,ndocs,nbits", [("tiny", None, 2), ("100k", 3000, 2), ("2m-long", 300, 4),
                                              ("1m", 3000, 2)])
def test_builder_matches_oracle(name, ndocs, nbits):
    w, c, k, cl = corpus(name, ndocs)
    oi = oracle_index(name, ndocs)
    b = product_builder(c, nbits, docs_per_chunk=700)
    cut, wb = b.quantizer()
    assert np.array_equal(cut, oi.cut_k)
    assert np.array_equal(wb, synth.k_to_bf16_bits(oi.w_k.astype(np.int16)))
    sec = b.sections()
    assert np.array_equal(sec["doc_off"], c.doc_off)
    assert np.array_equal(sec["cid"], cl)
    assert np.array_equal(sec["codes"], oracle.pack(oi.codes, nbits))
    assert np.array_equal(sec["ivf_off"], oi.ivf_off)
    assert np.array_equal(sec["ivf_doc"], oi.ivf_doc)
    inf = b.info()
    assert inf["ndocs"] == c.spec.ndocs and inf["ntokens"] == c.ntok and inf["max_doc_len"] == c.lengths.max()


def test_builder_rejects_bad_input():
    cent = np.zeros((4, 128), np.uint16)
    with pytest.raises(ChimeraError) as e:
        Builder(cent, 3)
    assert e.value.code == chimera.E_INVAL
    with pytest.raises(ChimeraError) as e:
        Builder(np.zeros((4, 64), np.uint16), 2)
    assert e.value.code == chimera.E_UNSUPPORTED
    b = Builder(cent, 2)
    with pytest.raises(ChimeraError):
        b.add_docs(np.zeros((1, 128), np.uint16), np.zeros(1, np.int32), np.ones(1, np.int32))  # not frozen
    with pytest.raises(ChimeraError):
        b.freeze()  # nothing added
    with pytest.raises(ChimeraError):
        b.add_residuals(np.zeros((1, 128), np.uint16), np.array([4], np.int32))  # cid out of range
    big = np.full((1, 128), 0x4000, np.uint16)  # 2.0 is outside [-1, 1]
    with pytest.raises(ChimeraError):
        b.add_residuals(big, np.zeros(1, np.int32))


def test_builder_binding_checks_row_counts():
    """The library reads as many rows as cids (pass 1) or sum(doc_lens) (pass
    2) says: the binding refuses arrays of another shape before the call."""
    b = Builder(np.zeros((4, 128), np.uint16), 2)
    tok = np.zeros((6, 128), np.uint16)
    for t, c in [(tok[:5], np.zeros(6, np.int32)), (tok[:, :64], np.zeros(6, np.int32)),
                 (tok, np.zeros((6, 1), np.int32))]:
        with pytest.raises(ValueError):
            b.add_residuals(t, c)
    b.add_residuals(tok, np.zeros(6, np.int32))
    b.freeze()
    for t, c, lens in [(tok, np.zeros(6, np.int32), [2, 3]), (tok, np.zeros(5, np.int32), [2, 4]),
                       (tok[:5], np.zeros(6, np.int32), [2, 4]), (tok, np.zeros(6, np.int32), [[2, 4]])]:
        with pytest.raises(ValueError):
            b.add_docs(t, c, np.array(lens, np.int32))
    b.add_docs(tok, np.zeros(6, np.int32), np.array([2, 4], np.int32))
    assert b.info()["ndocs"] == 2 and b.info()["ntokens"] == 6


def _read_header(path):
    raw = open(path, "rb").read()
    magic, ver, hb, dim, nbits, ncent, maxlen, ndocs, ntok, nnz, nsec = struct.unpack_from("<8sIIiiiiqqqI", raw, 0)
    secs = [struct.unpack_from("<IIQQQ", raw, 64 + 32 * i) for i in range(nsec)]
    return raw, dict(magic=magic, ver=ver, dim=dim, nbits=nbits, ncent=ncent, ndocs=ndocs, ntok=ntok, nnz=nnz), secs


def test_index_file_layout_and_corruption(tmp_path):
    w, c, k, cl = corpus("tiny")
    b = product_builder(c, 2)
    path = str(tmp_path / "tiny.chimidx")
    b.save(path)
    raw, hd, secs = _read_header(path)
    assert hd["magic"] == b"CHIMIDX1" and hd["ver"] == 1 and hd["ndocs"] == 1000 and hd["ntok"] == 32000
    sec = b.sections()
    # section 4 is the packed codes, section 8 the posting docs; offsets 256-B aligned
    for (sid, _, off, nbytes, _), arr in zip([secs[3], secs[7]], [sec["codes"], sec["ivf_doc"]]):
        assert off % 256 == 0 and raw[off:off + nbytes] == arr.tobytes()
    # loading validates before touching the GPU
    bad = bytearray(raw)
    bad[secs[3][2] + 5] ^= 0xFF
    p2 = str(tmp_path / "bad.chimidx")
    open(p2, "wb").write(bytes(bad))
    with pytest.raises(ChimeraError) as e:
        Index.load(p2)
    assert e.value.code == chimera.E_FORMAT and "checksum" in str(e.value)
    open(p2, "wb").write(raw[: len(raw) // 2])
    with pytest.raises(ChimeraError) as e:
        Index.load(p2)
    assert e.value.code == chimera.E_FORMAT
    bad = bytearray(raw)
    bad[8:12] = struct.pack("<I", 99)
    open(p2, "wb").write(bytes(bad))
    with pytest.raises(ChimeraError) as e:
        Index.load(p2)
    assert e.value.code == chimera.E_FORMAT and "version" in str(e.value)
    with pytest.raises(ChimeraError) as e:
        Index.load(str(tmp_path / "missing.chimidx"))
    assert e.value.code == chimera.E_IO
