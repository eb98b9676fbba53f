"""The transposed FP8 operands are K-blocked on the device: element (c, r) of the transpose of a
[rows, cols] tensor -- input row r, column c -- is at [r // 128, c, r % 128] of a
[rows // 128, cols, 128] buffer.  The oracle keeps the plain transpose [cols, rows]; these
convert between the two, for numpy arrays and torch tensors alike (no arithmetic)."""


def to_kblock(qT):
    """[cols, rows] -> [rows // 128, cols, 128]."""
    cols, rows = qT.shape
    v = qT.reshape(cols, rows // 128, 128)
    return v.permute(1, 0, 2).contiguous() if hasattr(v, "permute") else v.transpose(1, 0, 2).copy()


def from_kblock(qk):
    """[rows // 128, cols, 128] -> [cols, rows]."""
    nb, cols, _ = qk.shape
    v = qk.permute(1, 0, 2) if hasattr(qk, "permute") else qk.transpose(1, 0, 2)
    return v.reshape(cols, nb * 128)
