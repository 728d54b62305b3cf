"""Oracle of the hyper-decoder and the synthesis transform (TEST
INFRASTRUCTURE ONLY, like the rest of this package; it shares no code with
the GPU path).

The paper decodes pre-trained CompressAI models (Sec. IV-A; the latent
pipeline of Sec. II-A: z_hat -> hyper-decoder h_s -> entropy parameters,
y_hat -> synthesis transform g_s -> image).  It does not list their layers;
the layer list taken here is that of the mean-scale hyperprior model of the
Minnen et al. 2018 family the workloads are named after (N, M channels):

  h_s: transposed conv 5x5 stride 2 (N -> M), ReLU,
       transposed conv 5x5 stride 2 (M -> 3M/2), ReLU,
       conv 3x3 stride 1 (3M/2 -> 2M)                      -> psi [2M]
  g_s: three times transposed conv 5x5 stride 2 followed by inverse GDN
       (M -> N, N -> N, N -> N), then transposed conv 5x5 stride 2 (N -> 3)

Transposed convs use padding 2 and output padding 1 (each doubles the size),
the 3x3 conv padding 1.  Inverse GDN: out_c = x_c * sqrt(beta_c +
sum_j gamma_cj x_j^2).  Everything is plain PyTorch CPU in fp64 on NHWC
arrays (converted to NCHW around the library calls).
"""
import numpy as np
import torch
import torch.nn.functional as F


def _t(a):
    return torch.from_numpy(np.asarray(a, np.float64))


def deconv(x, w, b):
    """Transposed conv 5x5, stride 2, padding 2, output padding 1 (NCHW)."""
    return F.conv_transpose2d(x, _t(w), _t(b), stride=2, padding=2, output_padding=1)


def conv3(x, w, b):
    return F.conv2d(x, _t(w), _t(b), stride=1, padding=1)


def igdn(x, beta, gamma):
    """Inverse GDN over the channel axis of NCHW x."""
    z = torch.einsum("cj,njhw->nchw", _t(gamma), x * x) + _t(beta)[None, :, None, None]
    return x * torch.sqrt(z)


def _nchw(a):
    return torch.from_numpy(np.asarray(a, np.float64)).permute(0, 3, 1, 2)


def _nhwc(t):
    return t.permute(0, 2, 3, 1).contiguous().numpy()


def hyper_synthesis(z, w):
    """z_hat [B][Hz][Wz][N] -> psi [B][4Hz][4Wz][2M] (fp64)."""
    x = torch.relu(deconv(_nchw(z), w["hs1_w"], w["hs1_b"]))
    x = torch.relu(deconv(x, w["hs2_w"], w["hs2_b"]))
    return _nhwc(conv3(x, w["hs3_w"], w["hs3_b"]))


def synthesis(y, w):
    """y_hat [B][H][W][M] -> image [B][16H][16W][3] (fp64)."""
    x = _nchw(y)
    for k in (1, 2, 3):
        x = igdn(deconv(x, w[f"gs{k}_w"], w[f"gs{k}_b"]), w[f"gdn{k}_beta"], w[f"gdn{k}_gamma"])
    return _nhwc(deconv(x, w["gs4_w"], w["gs4_b"]))
