"""Host side of the trusted computing base: fail-closed policy resolution and the
per-row expansion of the decision into device policy words.

Sec. 3.1 (resolver paragraph) and App. B.1: only a trusted mapping whose
`allow_private` value has Boolean type and equals true allows; missing metadata,
wrong keys, strings, numbers, lists, nested values, nulls and serialized JSON text
all deny. The decision is expanded per batch row before routing (App. B.1), as one
32-bit word per token; the device allows only the single word PMPE_POLICY_ALLOW.
"""
from __future__ import annotations

from collections.abc import Mapping
from typing import Any, Sequence

import numpy as np
import torch

from ._native import PMPE_POLICY_ALLOW, PMPE_POLICY_DENY


def resolve_policy(meta: Any) -> bool:
    """True only for a mapping with allow_private of type bool equal to True."""
    if not isinstance(meta, Mapping) or "allow_private" not in meta:
        return False
    value = meta["allow_private"]
    return type(value) is bool and value is True


def policy_word(meta: Any) -> int:
    return PMPE_POLICY_ALLOW if resolve_policy(meta) else PMPE_POLICY_DENY


def token_policy_words(metas: Sequence[Any], lengths: Sequence[int], device=None) -> torch.Tensor:
    """uint32-valued words [T] (stored as int32 bit patterns): each request's word
    repeated over its rows."""
    words = np.repeat(np.asarray([policy_word(m) for m in metas], dtype=np.uint32),
                      np.asarray(lengths, dtype=np.int64))
    t = torch.from_numpy(words.view(np.int32).copy())
    return t if device is None else t.to(device)


def request_offsets(lengths: Sequence[int], device=None) -> torch.Tensor:
    off = np.concatenate([[0], np.cumsum(np.asarray(lengths, dtype=np.int64))]).astype(np.int32)
    t = torch.from_numpy(off)
    return t if device is None else t.to(device)
