"""Fixed codec tables, as data.

The paper fixes the *kind* of each table but prints none of their values:
  * a static table of 256 pseudo-random signs tiled over the coordinates
    (Section "Sign Flips and Dimension Permutation");
  * a static 128-element permutation applied within a block (same section);
  * Lloyd-Max codebooks for the standard normal distribution, 1-D with K=16
    (4-bit) and K=8 (3-bit), 2-D with K=16 (2-bit) and 4-D with K=16 (1-bit),
    obtained by k-means on synthetic N(0, I) samples
    (Section "Quantization Using Lloyd-Max Codebook", table tab:rslm_codecs).

Readings used here:
  * signs: ``numpy.random.default_rng(1).integers(0, 2, 256)``, 0 -> +1, 1 -> -1;
  * permutation: ``numpy.random.default_rng(2).permutation(128)``;
  * codebooks: produced once by ``synth/make_codebooks.py`` and stored in
    ``synth/codebooks.json`` with every centroid rounded to a value that
    float16 represents exactly (so a half-precision decode is lossless).
"""

import json
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_CODEBOOK_FILE = os.path.join(_HERE, "codebooks.json")
_cache = {}


def sign_table():
    """256 signs as int8 (+1/-1)."""
    bits = np.random.default_rng(1).integers(0, 2, 256)
    return np.where(bits == 0, 1, -1).astype(np.int8)


def permutation_table():
    """The 128-element intra-block permutation as int32."""
    return np.random.default_rng(2).permutation(128).astype(np.int32)


def _load():
    if "cb" not in _cache:
        with open(_CODEBOOK_FILE) as f:
            _cache["cb"] = json.load(f)
    return _cache["cb"]


def codebook(name):
    """Return a codebook as a (K, g) float32 array.

    ``name`` is a bit width (1, 2, 3, 4) for the codec codebooks, or one of
    the test-only 1-D tables ``"lm1d_k2"`` / ``"lm1d_k4"``.
    """
    key = {1: "rslm1", 2: "rslm2", 3: "rslm3", 4: "rslm4"}.get(name, name)
    rec = _load()[key]
    arr = np.asarray(rec["centroids"], dtype=np.float32)
    return arr.reshape(rec["K"], rec["g"])


def codebook_shape(name):
    rec = _load()[{1: "rslm1", 2: "rslm2", 3: "rslm3", 4: "rslm4"}.get(name, name)]
    return rec["K"], rec["g"]
